// The chain kernel of the LBI interface-adjoint scan on gfx950 (MI355X).
//
// Computes, for B independent chains of K slots,
//     (P_j, c_j) = (A_j, b_j) o (A_{j+1}, b_{j+1}) o ... o (A_{K-1}, b_{K-1}),
//     lambda_j   = P_j lambda_K + c_j,
// with the combine (A, b) o (A', b') = (A A', A b' + b) of the scan
// formulation (Proposition "Scan Formulation of Backpropagation"; Theorem
// "Bounded-Interface Backpropagation" gives lambda_j = mbar_j when b = 0), and
// Phase 2 of Algorithm "Bounded-Interface Backpropagation" (apply the suffix
// products to mbar_K, every slot).  A workgroup folds one segment of one
// chain: the whole chain (then it writes every lambda_j), or, in the
// two-level scan, a segment: first to its aggregate (the composite at its
// first slot), for the carry pass, then again from the segment's carry in
// place of lambda_K, writing its lambda_j.
//
// Kernel design (one workgroup per chain segment, NW waves):
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
//     bytes per lane, branch-free) -> LDS, one barrier per slot.  While a tile
//     is staged from registers, the same registers give the affine update
//     c_j = A_j c_{j+1} + b_j (partial dot products reduced across the lanes
//     that share a row), so A is never re-read for it.  Slot j-1 is staged
//     while the MFMAs of slot j run.
//   * The apply of slot j+1 (P_{j+1} lambda_K: per-wave partial sums reduced
//     by a DPP butterfly, then across waves through LDS) is issued between
//     the MFMAs that form P_j, so VALU and matrix-core work overlap;
//     lambda_j is stored once, coalesced, by one wave in turn.
//   * Three arithmetic modes:
//       kF32   fp32 storage, v_mfma_f32_16x16x4_f32;
//       kBF16  bf16 storage, v_mfma_f32_16x16x32_bf16; the fp32 composite is
//              fed back as bf16 hi + lo (two MFMAs), so the only bf16
//              rounding is the inputs';
//       kBF16R1  the same, with the composite fed back rounded once to bf16
//              (one MFMA): a relative error of about 2^-9 per slot, which
//              grows with the chain's length (opt-in);
//       kF32X  fp32 storage on the bf16 matrix cores: A_j and P are each cut
//              into three bf16 parts whose sum is exactly the fp32 value
//              (the value rounded to nearest, then its remainder, twice), and
//              the product keeps the six partial products down to 2^-16 of
//              the leading one, accumulated in fp32.  The parts are centred,
//              so the dropped products carry no bias; the error is at or
//              below that of fp32 MFMA, also over chains of hundreds of
//              slots that do not decay.
//     bf16 tiles sit in LDS with each 32-wide k block stored in MFMA operand
//     order, so one 16-byte LDS read yields a lane's 8 operand values.
//   * Widths hint: loads of all-zero tile regions are skipped (out-of-range
//     buffer offsets return zero without touching memory) and the combine
//     runs a shape specialised to the slot's row and k blocks.  The width
//     codes come from the kernel arguments through scalar loads, whose wait
//     also drains the LDS queue; the slot loop therefore keeps the codes of
//     the slots it touches in registers and fetches one new code per slot,
//     a slot early, where the slot barrier's wait covers it.
//
// All HIP code here is built with packed fp32 math disabled.
#ifndef LBI_CHAIN_HPP
#define LBI_CHAIN_HPP

#include <type_traits>

#include "lbi_device.hpp"
#include "lbi_internal.h"

namespace lbi {
namespace {

// E: storage element; L: LDS element of the staged A tile; PLANES: LDS
// copies of the tile (three bf16 parts for kF32X); PAD: row padding in L.
template <int M> struct Mode;
template <> struct Mode<kF32> {
    typedef float E;
    typedef float L;
    static constexpr int PLANES = 1, PAD = 4;
};
template <> struct Mode<kBF16> {
    typedef __bf16 E;
    typedef __bf16 L;
    static constexpr int PLANES = 1, PAD = 8;
};
template <> struct Mode<kBF16R1> : Mode<kBF16> {};
template <> struct Mode<kF32X> {
    typedef float E;
    typedef __bf16 L;
    static constexpr int PLANES = 3, PAD = 8;
};

__device__ __forceinline__ int width_blocks(const ScanArgs &a, int64_t k)
{
    return (int)((a.wcode[k >> 3] >> ((k & 7) * 4)) & 15u);
}

// Geometry shared by the kernel and its pieces.
template <int R, int M, int NCA> struct Geo {
    static constexpr int NW = waves_for(R);
    static constexpr int T = 64 * NW;
    static constexpr int NRB = R / 16;    // 16-row blocks
    static constexpr int CB = NCA / NW;   // column blocks per wave
    using E = typename Mode<M>::E;
    using L = typename Mode<M>::L;
    static constexpr int PLANES = Mode<M>::PLANES;
    static constexpr int ESZ = sizeof(E);
    static constexpr int PITCH = R + Mode<M>::PAD;               // LDS row pitch in L
    static constexpr bool PERM = sizeof(L) == 2 && R >= 32;      // k blocks in operand order
    static constexpr bool SWZ = PERM;                            // swizzled bf16 planes
    static constexpr int PLANE = SWZ ? R * R : R * PITCH;        // elements per LDS plane
    static constexpr int EPC = 16 / ESZ;                         // elements per 16-byte chunk
    static constexpr int TILE_CHUNKS = R * R / EPC;
    static constexpr int CPT = (TILE_CHUNKS + T - 1) / T;        // chunks per thread
    static constexpr int LPR = R / EPC;                          // staging lanes per tile row
    static constexpr int RPI = T / LPR;                          // tile rows per chunk index
    static constexpr int SHIFT_S = ilog2(LPR) - ilog2(CPT);      // staging reduce layout
    // slots prefetched (bf16 at r <= 32 takes a third; at r = 64 the third
    // costs the fifth wave per SIMD, which is worth more)
    static constexpr int NPF = ((M == kBF16 || M == kBF16R1) && R <= 32) ? 3 : 2;
    static constexpr int WPF = R > 64 ? R / 64 : 1;              // waves per finalize
    static constexpr int NWF = NW / WPF;                         // finalizing wave groups
    static_assert(NCA % NW == 0 && CB >= 1, "tile geometry");
    static_assert(CPT <= LPR && (T * EPC) % R == 0, "staging geometry");
};

// LDS column of tile column col (col % 4 == 0) in a k-permuted bf16 row: in
// each 32-wide block, operand lane group g reads k = 4g..4g+3 and
// 16+4g..16+4g+3 as its 8 consecutive values.
template <bool PERM> __device__ __forceinline__ int lds_col(int col)
{
    if constexpr (!PERM) {
        return col;
    } else {
        const int q = col & 31;
        return (col & ~31) + (((q & 15) >> 2) << 3) + ((q >> 4) << 2);
    }
}

// Element offset of (row, physical column pc) in a swizzled bf16 plane (R >=
// 32): rows hold C = R / 8 chunks of 16 bytes, 16 / C rows share a 256-byte
// line, and chunk q of row r sits in slot (r % (16 / C)) C + (q ^ (r / (16 / C)) % C).
// The 16 lanes that an access serves together then hit 16 distinct slots
// (all 64 banks), both for an operand read (one chunk of 16 consecutive rows)
// and for the staging writes (whole rows, 256 bytes at a time).
template <int R> __device__ __forceinline__ int swz_pos(int row, int pc)
{
    constexpr int C = R / 8, RHO = 16 / C;
    const int line = row / RHO, q = pc >> 3;
    return line * 128 + ((row % RHO) * C + (q ^ (line % C))) * 8 + (pc & 7);
}

// A operand (8 bf16 values) of row block I, k pair p, from one LDS plane.
template <int R, int PITCH>
__device__ __forceinline__ bf16x8 a_operand(const __bf16 *plane, int I, int p, int li, int g)
{
    if constexpr (R >= 32) {
        return *(const bf16x8 *)&plane[swz_pos<R>(16 * I + li, 32 * p + 8 * g)];
    } else {
        const bf16x4 a0 = *(const bf16x4 *)&plane[li * PITCH + 4 * g];
        const bf16x4 z = {};
        return __builtin_shufflevector(a0, z, 0, 1, 2, 3, 4, 5, 6, 7);
    }
}

struct NoFill {
    __device__ void operator()(int) const {}
};

// Pn = A_j * P on the matrix cores, for the first NR row blocks and NK k blocks
// (the rest of A_j is zero); rows past NR come out zero.  With FILL, fill(s)
// runs after MFMA group s of the split arithmetic (the six partial-product
// groups of each k pair), fenced so that the compiler keeps it there: other
// work placed in the shadow of the matrix cores.
template <int R, int M, int NCA, int NR, int NK, bool FILL = false, typename F = NoFill>
__device__ __forceinline__ void combine(f4 (&Pn)[R / 16][NCA / waves_for(R)],
                                        const f4 (&P)[R / 16][NCA / waves_for(R)],
                                        const typename Mode<M>::L *sAbuf, int li, int g,
                                        F &&fill = F())
{
    auto after_group = [&](int step) {
        if constexpr (FILL) {
            __builtin_amdgcn_sched_barrier(0);
            fill(step);
            __builtin_amdgcn_sched_barrier(0);
        }
    };
    using G = Geo<R, M, NCA>;
    constexpr int NRB = G::NRB, CB = G::CB, PITCH = G::PITCH;
    constexpr int PLANE = G::PLANE;
#pragma unroll
    for (int I = 0; I < NRB; ++I)
#pragma unroll
        for (int t = 0; t < CB; ++t)
            Pn[I][t] = f4{0.0f, 0.0f, 0.0f, 0.0f};
    if constexpr (M == kF32) {
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
        // k runs over pairs of 16-row blocks of P (operand value e < 4 from
        // the first block, e >= 4 from the second); a missing second block is
        // zero in both operands.
        constexpr int NKP = (NK + 1) / 2;
        constexpr bool kPairs = NRB >= 2;
#pragma unroll
        for (int p = 0; p < NKP; ++p) {
            float x[CB][8];
#pragma unroll
            for (int t = 0; t < CB; ++t)
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    x[t][v] = P[2 * p][t][v];
                    x[t][v + 4] = kPairs ? P[kPairs ? 2 * p + 1 : 0][t][v] : 0.0f;
                }
            if constexpr (M == kBF16R1) {
                // P rounded once to bf16 (RNE), two values per instruction
                bf16x8 bh[CB];
#pragma unroll
                for (int t = 0; t < CB; ++t) {
                    u4 hh;
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        hh[e] = __builtin_bit_cast(
                            uint32_t, __builtin_convertvector(f2{x[t][2 * e], x[t][2 * e + 1]}, bf16x2));
                    bh[t] = __builtin_bit_cast(bf16x8, hh);
                }
#pragma unroll
                for (int I = 0; I < NR; ++I) {
                    const bf16x8 a = a_operand<R, PITCH>(sAbuf, I, p, li, g);
#pragma unroll
                    for (int t = 0; t < CB; ++t)
                        Pn[I][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bh[t], Pn[I][t], 0, 0, 0);
                }
            } else if constexpr (M == kBF16) {
                // P = hi + lo (RNE hi, exact remainder, RNE lo), converted
                // two values per instruction
                bf16x8 bh[CB], bl[CB];
#pragma unroll
                for (int t = 0; t < CB; ++t) {
                    u4 hh, ll;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const uint32_t hu = __builtin_bit_cast(
                            uint32_t, __builtin_convertvector(f2{x[t][2 * e], x[t][2 * e + 1]}, bf16x2));
                        const f2 rest = {x[t][2 * e] - bitsf(hu << 16),
                                         x[t][2 * e + 1] - bitsf(hu & kHighHalf)};
                        hh[e] = hu;
                        ll[e] = __builtin_bit_cast(uint32_t, __builtin_convertvector(rest, bf16x2));
                    }
                    bh[t] = __builtin_bit_cast(bf16x8, hh);
                    bl[t] = __builtin_bit_cast(bf16x8, ll);
                }
#pragma unroll
                for (int I = 0; I < NR; ++I) {
                    const bf16x8 a = a_operand<R, PITCH>(sAbuf, I, p, li, g);
#pragma unroll
                    for (int t = 0; t < CB; ++t) {
                        Pn[I][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bh[t], Pn[I][t], 0, 0, 0);
                        Pn[I][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bl[t], Pn[I][t], 0, 0, 0);
                    }
                }
            } else {
                bf16x8 bh[CB], bm[CB], bl[CB];
#pragma unroll
                for (int t = 0; t < CB; ++t) {
                    u4 hh, mm, ll;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const Split2 s = split_pair_keep(x[t][2 * e], x[t][2 * e + 1]);
                        hh[e] = s.h;
                        mm[e] = s.m;
                        ll[e] = s.l;
                    }
                    bh[t] = __builtin_bit_cast(bf16x8, hh);
                    bm[t] = __builtin_bit_cast(bf16x8, mm);
                    bl[t] = __builtin_bit_cast(bf16x8, ll);
                }
                // the six partial products that reach 2^-16 of the leading one
                auto terms = [&](const bf16x8 &ah, const bf16x8 &am, const bf16x8 &al, f4 &acc,
                                 int t) {
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bh[t], acc, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bm[t], acc, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(am, bh[t], acc, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bl[t], acc, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, bh[t], acc, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(am, bm[t], acc, 0, 0, 0);
                };
                if constexpr (NR <= 4) {
                    // all operands first, then the products interleaved over
                    // the independent accumulators
                    bf16x8 ah[NR], am[NR], al[NR];
#pragma unroll
                    for (int I = 0; I < NR; ++I) {
                        ah[I] = a_operand<R, PITCH>(sAbuf, I, p, li, g);
                        am[I] = a_operand<R, PITCH>(sAbuf + PLANE, I, p, li, g);
                        al[I] = a_operand<R, PITCH>(sAbuf + 2 * PLANE, I, p, li, g);
                    }
#pragma unroll
                    for (int t = 0; t < CB; ++t)
#pragma unroll
                        for (int I = 0; I < NR; ++I)
                            Pn[I][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah[I], bh[t], Pn[I][t], 0, 0, 0);
                    after_group(6 * p + 0);
#pragma unroll
                    for (int t = 0; t < CB; ++t)
#pragma unroll
                        for (int I = 0; I < NR; ++I)
                            Pn[I][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah[I], bm[t], Pn[I][t], 0, 0, 0);
                    after_group(6 * p + 1);
#pragma unroll
                    for (int t = 0; t < CB; ++t)
#pragma unroll
                        for (int I = 0; I < NR; ++I)
                            Pn[I][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(am[I], bh[t], Pn[I][t], 0, 0, 0);
                    after_group(6 * p + 2);
#pragma unroll
                    for (int t = 0; t < CB; ++t)
#pragma unroll
                        for (int I = 0; I < NR; ++I)
                            Pn[I][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah[I], bl[t], Pn[I][t], 0, 0, 0);
                    after_group(6 * p + 3);
#pragma unroll
                    for (int t = 0; t < CB; ++t)
#pragma unroll
                        for (int I = 0; I < NR; ++I)
                            Pn[I][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al[I], bh[t], Pn[I][t], 0, 0, 0);
                    after_group(6 * p + 4);
#pragma unroll
                    for (int t = 0; t < CB; ++t)
#pragma unroll
                        for (int I = 0; I < NR; ++I)
                            Pn[I][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(am[I], bm[t], Pn[I][t], 0, 0, 0);
                    after_group(6 * p + 5);
                } else {
#pragma unroll
                    for (int I = 0; I < NR; ++I) {
                        const bf16x8 ah = a_operand<R, PITCH>(sAbuf, I, p, li, g);
                        const bf16x8 am = a_operand<R, PITCH>(sAbuf + PLANE, I, p, li, g);
                        const bf16x8 al = a_operand<R, PITCH>(sAbuf + 2 * PLANE, I, p, li, g);
#pragma unroll
                        for (int t = 0; t < CB; ++t)
                            terms(ah, am, al, Pn[I][t], t);
                    }
                }
            }
        }
    }
}

// Runtime (row blocks, k blocks) of a hinted slot -> the specialised combine
// for the next powers of two (extra blocks multiply zeros).
template <int R, int M, int NCA, int NR>
__device__ __forceinline__ void combine_k(int nk, f4 (&Pn)[R / 16][NCA / waves_for(R)],
                                          const f4 (&P)[R / 16][NCA / waves_for(R)],
                                          const typename Mode<M>::L *sAbuf, int li, int g)
{
    constexpr int NRB = R / 16;
    if (nk <= 1 || NRB == 1) { combine<R, M, NCA, NR, 1>(Pn, P, sAbuf, li, g); return; }
    if constexpr (NRB >= 2) if (nk <= 2) { combine<R, M, NCA, NR, 2>(Pn, P, sAbuf, li, g); return; }
    if constexpr (NRB >= 4) if (nk <= 4) { combine<R, M, NCA, NR, 4>(Pn, P, sAbuf, li, g); return; }
    if constexpr (NRB >= 8) combine<R, M, NCA, NR, 8>(Pn, P, sAbuf, li, g);
}

template <int R, int M, int NCA>
__device__ __forceinline__ void combine_shape(int nr, int nk, f4 (&Pn)[R / 16][NCA / waves_for(R)],
                                              const f4 (&P)[R / 16][NCA / waves_for(R)],
                                              const typename Mode<M>::L *sAbuf, int li, int g)
{
    constexpr int NRB = R / 16;
    if (nr <= 1 || NRB == 1) { combine_k<R, M, NCA, 1>(nk, Pn, P, sAbuf, li, g); return; }
    if constexpr (NRB >= 2) if (nr <= 2) { combine_k<R, M, NCA, 2>(nk, Pn, P, sAbuf, li, g); return; }
    if constexpr (NRB >= 4) if (nr <= 4) { combine_k<R, M, NCA, 4>(nk, Pn, P, sAbuf, li, g); return; }
    if constexpr (NRB >= 8) combine_k<R, M, NCA, 8>(nk, Pn, P, sAbuf, li, g);
}

template <int R, int M, bool AFF, int HINT, int NCA, int OUT>
__global__ __launch_bounds__(64 * waves_for(R)) void scan_chain_kernel(const ScanArgs args)
{
    static_assert(OUT == kOutLambda || NCA == R / 16, "composites are written whole");
    using G = Geo<R, M, NCA>;
    using E = typename G::E;
    using L = typename G::L;
    constexpr int NW = G::NW, T = G::T, NRB = G::NRB, CB = G::CB;
    constexpr int PITCH = G::PITCH, EPC = G::EPC, CPT = G::CPT;
    constexpr int TILE_CHUNKS = G::TILE_CHUNKS, LPR = G::LPR, RPI = G::RPI;
    constexpr int SHIFT_S = G::SHIFT_S, PLANES = G::PLANES;
    constexpr bool PERM = G::PERM;
    constexpr int NPF = G::NPF, WPF = G::WPF, NWF = G::NWF;
    constexpr int TILE_BYTES = R * R * G::ESZ;
    constexpr int PLANE = G::PLANE;
    // element offset of (row, physical column) in an LDS plane
    auto tpos = [](int row, int pc) {
        if constexpr (G::SWZ)
            return swz_pos<R>(row, pc);
        else
            return row * PITCH + pc;
    };

    __shared__ __attribute__((aligned(16))) L sA[2][PLANES * PLANE];
    // c_s in a ring of four, indexed (K - s) mod 4
    __shared__ __attribute__((aligned(16))) float sC[AFF ? 4 : 1][R];
    __shared__ __attribute__((aligned(16))) float sPart[OUT == kOutLambda ? 2 : 1][NW][R];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = tid >> 6;
    const int g = lane >> 4;
    const int li = lane & 15;
    // this workgroup's segment: slots s0 .. s0 + K - 1 of chain beta; below,
    // slot indices are local to the segment
    const int64_t beta = blockIdx.x / args.S;
    const int64_t s0 = (int64_t)(blockIdx.x % args.S) * args.L;
    const int64_t K = args.K - s0 < args.L ? args.K - s0 : args.L;
    const int64_t first = beta * args.K + s0;  // global index of local slot 0
    // compact storage (hinted whole chains): per-chain bases, and running
    // element offsets of the A, b and lambda streams, each walked from the
    // chain's end one slot at a time (every stream visits slots K-1, K-2, ...)
    constexpr bool compact = HINT == kHintCompact && OUT == kOutLambda;
    const E *A = (const E *)args.A +
                 (compact ? beta * (int64_t)args.totalA : first * (int64_t)(R * R));
    const E *bv = AFF ? (const E *)args.b + (compact ? beta * (int64_t)args.totalR
                                                     : first * (int64_t)R)
                      : nullptr;
    float *lam = OUT == kOutLambda
                     ? args.lam + (compact ? beta * (int64_t)args.totalR : first * (int64_t)R)
                     : nullptr;
    int32_t curA = args.totalA, curB = args.totalR, curL = args.totalR;
    // (compact: one buffer resource per stream and chain; the running offset
    // goes in the scalar offset of each access)
    const __amdgpu_buffer_rsrc_t rsA_c = __builtin_amdgcn_make_buffer_rsrc(
        (void *)A, 0, compact ? args.totalA * G::ESZ : 0, kBufferWord3);
    // composites at [B][K], or only the segment aggregates at [B][S]
    const int64_t cslot = args.agg_only ? (int64_t)blockIdx.x : first;
    float *Pout = OUT == kOutComposite ? args.Pout + cslot * (int64_t)(R * R) : nullptr;
    float *cout = OUT == kOutComposite ? args.cout : nullptr;  // NULL: not written
    if (cout)
        cout += cslot * (int64_t)R;
    auto ring = [&](int64_t s) { return (int)((K - s) & 3); };
    // width code of local slot x (its row blocks; x = K: lambda_K's), 0
    // before the segment.  The slot loop keeps the codes it needs in a
    // rolling window instead (see below): each lookup is a scalar load, whose
    // wait also drains the LDS queue.
    auto wlook = [&](int64_t x) -> int {
        if constexpr (HINT)
            return x >= 0 ? width_blocks(args, s0 + x) : 0;
        else
            return 0;
    };
    // rows of a slot with width code wc that can be nonzero, rounded up to
    // 16 x a power of two
    auto rows_of = [&](int wc) {
        if constexpr (HINT)
            return 16 * pow2_at_least(wc);
        else
            return R;
    };
    auto live_rows = [&](int64_t s) {
        if constexpr (HINT)
            return s >= 0 && s < K ? rows_of(wlook(s)) : 0;
        else
            return R;
    };

    // staging lane roles: chunk i of this thread covers tile row
    // i * RPI + srow, columns scol .. scol + EPC - 1; after the row reduce,
    // this lane owns the affine sum of row orow (if oown)
    const int sgi = tid % LPR;
    const int srow = tid / LPR;
    const int scol = sgi * EPC;
    const int orow = (sgi >> SHIFT_S) * RPI + srow;
    const bool oown = (sgi & ((1 << SHIFT_S) - 1)) == 0 && orow < R;

    // ---- staging: HBM -> registers -> LDS -------------------------------------
    // Loads are issued unconditionally (a slot that does not exist gets only
    // out-of-range offsets), so the compiler can count outstanding loads
    // exactly and wait only for the slot being stored.
    // (wr, wc: width codes of slots j and j + 1, read with a widths hint)
    auto load_tile = [&](u4 (&dst)[CPT], int64_t j, bool valid, int wr, int wc) {
        const int64_t jj = valid ? j : 0;
        int rows = valid ? R : 0, cols = R;
        if constexpr (HINT) {
            rows = valid ? 16 * wr : 0;
            cols = 16 * wc;
        }
        if constexpr (compact) {
            // the r_j x r_{j+1} tile sits just below the previous one
            // (chunk i of this lane: row i * RPI + srow, columns scol ..; the
            // lane part of the offset is the same for every chunk, the row
            // step goes in the scalar offset)
            if (valid)
                curA -= rows * cols;
            const int vbase = (srow * cols + scol) * G::ESZ;
            const bool colok = scol < cols;
#pragma unroll
            for (int i = 0; i < CPT; ++i) {
                const int c = i * T + tid;
                const bool ok = c < TILE_CHUNKS && colok && i * RPI + srow < rows;
                dst[i] = __builtin_amdgcn_raw_buffer_load_b128(
                    rsA_c, ok ? vbase : kOutOfRange, (curA + i * RPI * cols) * G::ESZ, 0);
            }
        } else {
            const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
                (void *)(A + jj * (int64_t)(R * R)), 0, TILE_BYTES, kBufferWord3);
#pragma unroll
            for (int i = 0; i < CPT; ++i) {
                const int c = i * T + tid;
                const int e = c * EPC;
                const bool ok = c < TILE_CHUNKS && (e / R) < rows && (e % R) < cols;
                dst[i] = __builtin_amdgcn_raw_buffer_load_b128(rs, ok ? c * 16 : kOutOfRange, 0, 0);
            }
        }
    };
    // b_j at the row this lane owns after the staging reduce (raw bits)
    auto load_b = [&](int64_t j, bool valid, int wr) -> uint32_t {
        if constexpr (AFF) {
            int nrow = R, soff = 0;
            const E *base = bv + (valid ? j : 0) * (int64_t)R;
            int range = R * G::ESZ;
            if constexpr (compact) {
                // one resource over the chain's b; b_j just below b_{j+1}
                nrow = valid ? 16 * wr : 0;
                curB -= nrow;
                base = bv;
                range = args.totalR * G::ESZ;
                soff = curB * G::ESZ;
            }
            const __amdgpu_buffer_rsrc_t rs =
                __builtin_amdgcn_make_buffer_rsrc((void *)base, 0, range, kBufferWord3);
            const int off = (valid && oown && orow < nrow) ? orow * G::ESZ : kOutOfRange;
            if constexpr (G::ESZ == 4)
                return __builtin_amdgcn_raw_buffer_load_b32(rs, off, soff, 0);
            else
                return (uint32_t)__builtin_amdgcn_raw_buffer_load_b16(rs, off, soff, 0) << 16;
        } else {
            return 0u;
        }
    };
    // Tile j from registers into LDS buffer buf, and (affine) c_j = A_j c_{j+1}
    // + b_j from the same registers (c_{j+1} = 0 for the first slot).  In
    // three parts, so that the chunks can be spread between MFMAs.
    float st_cv[EPC];
    float st_part[CPT];
    auto stage_begin = [&](int64_t j, bool first) {
        if constexpr (AFF) {
#pragma unroll
            for (int e = 0; e < EPC; e += 4) {
                const f4 c4 = first ? f4{0.0f, 0.0f, 0.0f, 0.0f}
                                    : *(const f4 *)&sC[ring(j + 1)][scol + e];
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    st_cv[e + u] = c4[u];
            }
        }
    };
    // (lr: live rows of slot j, with a widths hint)
    auto stage_chunk = [&](const u4 &src, int i, int buf, int64_t j, int lr) {
        const int c = i * T + tid;
        const int row = i * RPI + srow;
        float x[EPC];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            if constexpr (G::ESZ == 4) {
                x[e] = bitsf(src[e]);
            } else {
                x[2 * e] = bitsf(src[e] << 16);
                x[2 * e + 1] = bitsf(src[e] & kHighHalf);
            }
        }
        if constexpr (AFF) {
            // with a widths hint, chunk rows at or past r_j are all zero
            float s = 0.0f;
            if (!HINT || i * RPI < lr) {
                s = x[0] * st_cv[0];
#pragma unroll
                for (int e = 1; e < EPC; ++e)
                    s += x[e] * st_cv[e];
            }
            st_part[i] = s;
        }
        if (TILE_CHUNKS % T == 0 || c < TILE_CHUNKS) {
            L *dst = sA[buf];
            if constexpr (M == kF32) {
                *(u4 *)&dst[tpos(row, scol)] = src;
            } else if constexpr (M == kBF16 || M == kBF16R1) {
                if constexpr (PERM) {
                    *(u2 *)&dst[tpos(row, lds_col<PERM>(scol))] = u2{src[0], src[1]};
                    *(u2 *)&dst[tpos(row, lds_col<PERM>(scol + 4))] = u2{src[2], src[3]};
                } else {
                    *(u4 *)&dst[tpos(row, scol)] = src;
                }
            } else {
                const Split2 s01 = split_pair(x[0], x[1]);
                const Split2 s23 = split_pair(x[2], x[3]);
                const int pos = tpos(row, lds_col<PERM>(scol));
                *(u2 *)&dst[pos] = u2{s01.h, s23.h};
                *(u2 *)&dst[PLANE + pos] = u2{s01.m, s23.m};
                *(u2 *)&dst[2 * PLANE + pos] = u2{s01.l, s23.l};
            }
        }
    };
    auto stage_end = [&](uint32_t braw, int64_t j) {
        if constexpr (AFF) {
            group_reduce<LPR, CPT>(st_part, sgi);
            if (oown)
                sC[ring(j)][orow] = st_part[0] + bitsf(braw);
        }
    };
    auto stage = [&](const u4 (&src)[CPT], int buf, uint32_t braw, int64_t j, bool first,
                     int lr) {
        stage_begin(j, first);
#pragma unroll
        for (int i = 0; i < CPT; ++i)
            stage_chunk(src[i], i, buf, j, lr);
        stage_end(braw, j);
    };

    // ---- per-lane constants ---------------------------------------------------
    float lk[CB];
    {
        // compact: lambda_K holds r_K values per chain
        const int rK = compact ? 16 * width_blocks(args, args.K) : R;
#pragma unroll
        for (int t = 0; t < CB; ++t) {
            const int idx = 16 * (w + NW * t) + li;
            // (segments: lambda at this segment's end, from the carry pass)
            lk[t] = OUT != kOutLambda || idx >= rK ? 0.0f
                    : args.lamSeg ? args.lamSeg[(int64_t)blockIdx.x * R + idx]
                                  : to_f32(((const E *)args.lamK)[beta * rK + idx]);
        }
    }

    // ---- the apply: partial P lambda_K over this wave's columns ---------------
    // (NB row blocks; with a widths hint, only the blocks slot s can fill)
    auto apply_rows = [&](const f4(&P)[NRB][CB], int pbuf, auto nb_tag) {
        constexpr int NB = decltype(nb_tag)::value;
        constexpr int VV = 4 * NB;
        constexpr int VFF = VV >= 16 ? VV / 16 : 1;
        constexpr int SH = VV >= 16 ? 0 : (VV == 8 ? 1 : 2);
        float q[VV];
#pragma unroll
        for (int I = 0; I < NB; ++I)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                float s = P[I][0][v] * lk[0];
#pragma unroll
                for (int t = 1; t < CB; ++t)
                    s += P[I][t][v] * lk[t];
                q[4 * I + v] = s;
            }
        group_reduce<16, VV>(q, li);
        if ((li & ((1 << SH) - 1)) == 0) {
#pragma unroll
            for (int e = 0; e < VFF; ++e) {
                const int idx = (li >> SH) * VFF + e;  // = 4*I + v
                const int row = 16 * (idx >> 2) + 4 * g + (idx & 3);
                sPart[pbuf][w][row] = q[e];
            }
        }
    };
    // (lr: live rows of slot s, with a widths hint)
    auto apply_partial = [&](const f4(&P)[NRB][CB], int pbuf, int64_t s, int lr) {
        if constexpr (HINT) {
            const int nb = lr / 16;
            if (nb <= 1 || NRB == 1) {
                apply_rows(P, pbuf, std::integral_constant<int, 1>{});
                return;
            }
            if constexpr (NRB >= 2)
                if (nb <= 2) {
                    apply_rows(P, pbuf, std::integral_constant<int, 2>{});
                    return;
                }
            if constexpr (NRB >= 4)
                if (nb <= 4) {
                    apply_rows(P, pbuf, std::integral_constant<int, 4>{});
                    return;
                }
            if constexpr (NRB >= 8)
                apply_rows(P, pbuf, std::integral_constant<int, 8>{});
        } else {
            apply_rows(P, pbuf, std::integral_constant<int, NRB>{});
        }
    };
    // ---- streaming: slots after which progress is published --------------------
    // every pchunk final slots, and the last one.  Slots are finalized in the
    // order K-1, K-2, ..., so a countdown over the finalized slots decides it
    // (finalize(x) sets pub_now; the publish_before(x) that follows it uses it).
    int32_t pub_left = args.pchunk;
    bool pub_now = false;
    // Called after a barrier that follows finalize(x): the storing wave group
    // fenced its stores of slots x .. K-1 before it, so the count K - x can be
    // published.
    // The count is raised with a system-scope atomic, so that it lands in
    // memory rather than in this XCD's L2: agents outside the XCD (another
    // XCD's waves, the command processor) poll it there.  With pub_clock the
    // same lane then records the real-time counter of the publication.
    auto publish_before = [&](int64_t x) {
        if constexpr (OUT == kOutLambda) {
            if (args.progress && pub_now && tid == 0) {
                const uint32_t n = (uint32_t)(K - x);
                __hip_atomic_fetch_max(&args.progress[beta], n, __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_SYSTEM);
                if (args.pub_clock)
                    args.pub_clock[beta * args.npub + (n + args.pchunk - 1) / args.pchunk - 1] =
                        __builtin_amdgcn_s_memrealtime();
            }
            pub_now = false;
        }
    };
    // ---- lambda_s = sum of the wave partials + c_s, stored by one wave group ---
    // Branch-free: lanes with nothing to store (and calls with valid = false)
    // get an out-of-range offset, which the buffer store drops; every wave
    // then issues the same memory instructions, which keeps the compiler's
    // count of outstanding loads exact.
    // (ws: width code of slot s, with a widths hint)
    auto finalize = [&](int64_t s, bool valid, int pbuf, int ws) {
        const int64_t ss = valid ? s : 0;
        // (when streaming, one wave group stores every slot, so that only it
        // has to fence before a publication)
        const int fw = args.progress ? 0 : (int)((uint64_t)ss % NWF);
        const int ft = tid - fw * 64 * WPF;
        const bool mine = valid && ft >= 0 && ft < R;
        const int fi = mine ? ft : 0;
        // rows the apply did not write are zero rows of P_s
        float acc = 0.0f;
        if (fi < (HINT ? (valid ? rows_of(ws) : 0) : R)) {
            acc = sPart[pbuf][0][fi];
#pragma unroll
            for (int ww = 1; ww < NW; ++ww)
                acc += sPart[pbuf][ww][fi];
        }
        if constexpr (AFF)
            acc += sC[ring(ss)][fi];
        // compact: lambda_s holds r_s values, just below lambda_{s+1}
        int nrow = R, soff = 0;
        float *base = lam + ss * R;
        int range = R * (int)sizeof(float);
        if constexpr (compact) {
            // one resource over the chain's lambda; lambda_s just below lambda_{s+1}
            nrow = valid ? 16 * ws : 0;
            curL -= nrow;
            base = lam;
            range = args.totalR * (int)sizeof(float);
            soff = curL * (int)sizeof(float);
        }
        const __amdgpu_buffer_rsrc_t rs =
            __builtin_amdgcn_make_buffer_rsrc((void *)base, 0, range, kBufferWord3);
        __builtin_amdgcn_raw_buffer_store_b32(
            __float_as_uint(acc), rs, mine && fi < nrow ? fi * (int)sizeof(float) : kOutOfRange,
            soff, 0);
        // Streaming: at a publish point the storing wave group makes its
        // lambda stores visible device-wide (release: L2 written back); after
        // the next barrier one lane raises progress[beta] to the count of
        // final adjoints (see publish_before).
        if constexpr (OUT == kOutLambda) {
            if (args.progress && valid) {
                pub_now = --pub_left == 0 || ss == 0;
                if (pub_left == 0)
                    pub_left = args.pchunk;
                if (pub_now && w / WPF == 0)
                    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
            }
        }
    };
    // ---- the composite (P_s, c_s) of local slot s, to global memory -----------
    // (branch-free buffer stores; each lane writes its rows of its columns)
    auto store_composite = [&](const f4 (&P)[NRB][CB], int64_t s) {
        if constexpr (OUT == kOutComposite) {
            if (args.agg_only && s != 0)
                return;
            const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
                (void *)(Pout + s * (int64_t)(R * R)), 0, R * R * (int)sizeof(float), kBufferWord3);
#pragma unroll
            for (int I = 0; I < NRB; ++I)
#pragma unroll
                for (int t = 0; t < CB; ++t)
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        const int row = 16 * I + 4 * g + v, col = 16 * (w + NW * t) + li;
                        __builtin_amdgcn_raw_buffer_store_b32(fbits(P[I][t][v]), rs,
                                                              (row * R + col) * (int)sizeof(float), 0, 0);
                    }
            if (cout) {
                // c_s (zero without an affine term)
                const __amdgpu_buffer_rsrc_t rc = __builtin_amdgcn_make_buffer_rsrc(
                    (void *)(cout + s * (int64_t)R), 0, R * (int)sizeof(float), kBufferWord3);
                const float cv = AFF ? sC[AFF ? ring(s) : 0][tid < R ? tid : 0] : 0.0f;
                __builtin_amdgcn_raw_buffer_store_b32(
                    fbits(cv), rc, tid < R ? tid * (int)sizeof(float) : kOutOfRange, 0, 0);
            }
        }
    };

    // ---- slot K-1: P = A_{K-1}, c = b_{K-1}; then stage slot K-2 --------------
    // Slot x is prefetched into register set (K-1-x) mod NPF and staged into
    // LDS buffer (K-1-x) mod 2.
    u4 pf[NPF][CPT];
    uint32_t pfb[NPF];
    {
        u4 first[CPT];
        const uint32_t firstb = load_b(K - 1, true, wlook(K - 1));
        load_tile(first, K - 1, true, wlook(K - 1), wlook(K));
#pragma unroll
        for (int q = 1; q <= NPF; ++q) {
            pfb[q % NPF] = load_b(K - 1 - q, K - 1 - q >= 0, wlook(K - 1 - q));
            load_tile(pf[q % NPF], K - 1 - q, K - 1 - q >= 0, wlook(K - 1 - q), wlook(K - q));
        }
        stage(first, 0, firstb, K - 1, true, live_rows(K - 1));
    }
    __syncthreads();

    f4 P[NRB][CB];
#pragma unroll
    for (int I = 0; I < NRB; ++I)
#pragma unroll
        for (int t = 0; t < CB; ++t)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int row = 16 * I + 4 * g + v, col = 16 * (w + NW * t) + li;
                const int pos = tpos(row, lds_col<PERM>(col & ~3) + (col & 3));
                if constexpr (M == kF32X)
                    P[I][t][v] = (to_f32(sA[0][pos]) + to_f32(sA[0][PLANE + pos])) +
                                 to_f32(sA[0][2 * PLANE + pos]);
                else
                    P[I][t][v] = to_f32(sA[0][pos]);
            }
    if (K >= 2) {
        stage(pf[1 % NPF], 1, pfb[1 % NPF], K - 2, false, live_rows(K - 2));
        pfb[1 % NPF] = load_b(K - 2 - NPF, K - 2 - NPF >= 0, wlook(K - 2 - NPF));
        load_tile(pf[1 % NPF], K - 2 - NPF, K - 2 - NPF >= 0, wlook(K - 2 - NPF),
                  wlook(K - 1 - NPF));
    }

    // ---- slots K-2 .. 0 ---------------------------------------------------------
    // Iteration j (A_j and c_j staged before its barrier): finalize slot j+2,
    // then the MFMAs of P_j = A_j P_{j+1} with, in their shadow, the staging
    // of slot j-1 (into the other LDS buffer; c_{j-1} from c_j) and the apply
    // of slot j+1.  One barrier per slot: the buffer staged here was last
    // read by the previous iteration's MFMAs, and c_{j-1} overwrites c_{j+3}
    // in the ring of four, whose readers all ran before this barrier.
    //
    // With a widths hint, wq[d] holds the width code of slot j + 2 - d
    // (d = 0 .. NPF + 3: every slot the iteration touches).  The window moves
    // by one slot per iteration; the code it takes in is looked up an
    // iteration early, before the barrier, whose wait covers the load.
    int wq[NPF + 4];
#pragma unroll
    for (int d = 0; d < NPF + 4; ++d)
        wq[d] = wlook(K - d);
    for (int64_t base = K - 2; base >= 0; base -= NPF) {
#pragma unroll
        for (int s = 0; s < NPF; ++s) {
            const int64_t j = base - s;
            if (j < 0)
                break;
            const int buf = (int)((uint32_t)(K - 1 - j) & 1);
            const int nx = (s + 2) % NPF;  // register set of slot j-1 (constant once unrolled)
            const int wnext = wlook(j - 2 - NPF);
            __syncthreads();
            publish_before(j + 3);
            if constexpr (OUT == kOutLambda)
                finalize(j + 2, j + 2 <= K - 1, (int)((j + 2) & 1), wq[0]);
            const int lr_next = j - 1 >= 0 ? rows_of(wq[3]) : 0;  // live rows of slot j-1
            f4 Pn[NRB][CB];
            // The staging of slot j-1 below is unconditional: at j = 0 it
            // stages the all-zero registers of the nonexistent slot -1 into a
            // buffer nothing reads again, and its c lands in ring entry
            // (K + 1) mod 4, which no later reader uses.
            auto reload = [&]() {
                pfb[nx] = load_b(j - 1 - NPF, j - 1 - NPF >= 0, wq[NPF + 3]);
                load_tile(pf[nx], j - 1 - NPF, j - 1 - NPF >= 0, wq[NPF + 3], wq[NPF + 2]);
            };
            auto emit = [&]() {
                if constexpr (OUT == kOutLambda)
                    apply_partial(P, (int)((j + 1) & 1), j + 1, rows_of(wq[1]));
                else
                    store_composite(P, j + 1);
            };
            if constexpr (M == kF32X && !HINT) {
                // split arithmetic: the staging chunks, the loads and the
                // apply go between the 6 (r = 16, 32) or 12 (r = 64) MFMA
                // groups of the combine
                // (the wave in its combine issues ahead of the other wave on
                // its SIMD: measured 0.6-1.4% faster on 512 chains of 512)
                __builtin_amdgcn_s_setprio(2);
                stage_begin(j - 1, false);
                combine<R, M, NCA, NRB, NRB, true>(Pn, P, sA[buf], li, g, [&](int step) {
                    if (step < CPT)
                        stage_chunk(pf[nx][step], step, buf ^ 1, j - 1, lr_next);
                    else if (step == CPT)
                        stage_end(pfb[nx], j - 1);
                    else if (step == CPT + 1)
                        reload();
                    else if (step == CPT + 2)
                        emit();
                });
                __builtin_amdgcn_s_setprio(0);
            } else {
                if constexpr (HINT) {
                    combine_shape<R, M, NCA>(pow2_at_least(wq[2]), pow2_at_least(wq[1]), Pn, P,
                                             sA[buf], li, g);
                } else {
                    combine<R, M, NCA, NRB, NRB>(Pn, P, sA[buf], li, g);
                }
                stage(pf[nx], buf ^ 1, pfb[nx], j - 1, false, lr_next);
                reload();
                emit();
            }
#pragma unroll
            for (int I = 0; I < NRB; ++I)
#pragma unroll
                for (int t = 0; t < CB; ++t)
                    P[I][t] = Pn[I][t];
#pragma unroll
            for (int d = 0; d < NPF + 3; ++d)
                wq[d] = wq[d + 1];
            wq[NPF + 3] = wnext;
        }
    }
    if constexpr (OUT == kOutLambda) {
        // slot 0's partials reuse the buffer finalize(2) read in the last
        // iteration
        __syncthreads();
        publish_before(2);
        apply_partial(P, 0, 0, live_rows(0));
        __syncthreads();
        finalize(1, K >= 2, 1, wlook(1));
        if (args.progress) {
            __syncthreads();
            publish_before(1);
        }
        finalize(0, true, 0, wlook(0));
        if (args.progress) {
            __syncthreads();
            publish_before(0);
        }
    } else {
        // c_0 was staged before the last barrier
        store_composite(P, 0);
    }
}


// ---- launch -----------------------------------------------------------------

template <int R, int M, bool AFF, int HINT, int NCA, int OUT>
hipError_t launch_kernel(const ChainLaunch &c)
{
    void *params[] = {(void *)&c.args};
    const int64_t grid = c.B * c.args.S;
    return hipLaunchKernel((const void *)&scan_chain_kernel<R, M, AFF, HINT, NCA, OUT>,
                           dim3((unsigned)grid), dim3(64 * waves_for(R)), params, 0, c.stream);
}

template <int M, bool AFF, int HINT, int OUT>
hipError_t launch_r(const ChainLaunch &c)
{
    switch (c.r) {
    case 16: return launch_kernel<16, M, AFF, HINT, 1, OUT>(c);
    case 32: return launch_kernel<32, M, AFF, HINT, 2, OUT>(c);
    case 64: return launch_kernel<64, M, AFF, HINT, 4, OUT>(c);
    default:
        if constexpr (M == kF32X) {
            // three bf16 planes of a 128-wide tile do not fit LDS twice over;
            // the host sends r = 128 fp32 work to the fp32 matrix cores
            return hipErrorInvalidValue;
        } else {
            // With a hint whose r_K <= 64 only the first four column blocks
            // of P can be nonzero (lambda output only).
            if constexpr (OUT == kOutLambda && HINT) {
                if (c.ncol <= 4)
                    return launch_kernel<128, M, AFF, HINT, 4, OUT>(c);
            }
            return launch_kernel<128, M, AFF, HINT, 8, OUT>(c);
        }
    }
}

template <int M>
hipError_t launch_chain(const ChainLaunch &c)
{
    if (c.out == kOutComposite) {
        if (c.aff)
            return c.hint ? launch_r<M, true, kHintWidths, kOutComposite>(c)
                          : launch_r<M, true, kHintNone, kOutComposite>(c);
        return c.hint ? launch_r<M, false, kHintWidths, kOutComposite>(c)
                      : launch_r<M, false, kHintNone, kOutComposite>(c);
    }
    if (c.hint && c.args.compact)
        return c.aff ? launch_r<M, true, kHintCompact, kOutLambda>(c)
                     : launch_r<M, false, kHintCompact, kOutLambda>(c);
    if (c.aff)
        return c.hint ? launch_r<M, true, kHintWidths, kOutLambda>(c)
                      : launch_r<M, true, kHintNone, kOutLambda>(c);
    return c.hint ? launch_r<M, false, kHintWidths, kOutLambda>(c)
                  : launch_r<M, false, kHintNone, kOutLambda>(c);
}

}  // namespace
}  // namespace lbi

#endif  // LBI_CHAIN_HPP
