// The chain scan with one wavefront per chain, for bf16 storage and r <= 64.
//
// It computes what the workgroup chain kernel computes (the suffix composites
// P_j = A_j P_{j+1} on the bf16 matrix cores, with the fp32 composite fed back
// as bf16 hi + lo; c_j = A_j c_{j+1} + b_j; lambda_j = P_j lambda_K + c_j, the
// apply of Algorithm "Bounded-Interface Backpropagation", Phase 2), mapped for
// many chains (a batch of token positions): one 64-lane wave owns a chain, so
// there is no barrier, no LDS staging of A and no reduction across waves.
//
//   * The wave holds all of P (R x R, fp32) in the accumulator layout of
//     v_mfma_f32_16x16x32_bf16: lane (g, li) = (lane / 16, lane % 16) holds
//     rows 16 I + 4 g + v (v < 4) of column 16 cb + li, for every row block I
//     and column block cb.  Read as a B operand, k pair p of column block cb
//     is rows 32 p + 4 g + v and 32 p + 16 + 4 g + v of that column.
//   * A_j goes from memory straight into A-operand registers in that k order:
//     for row block I and k pair p, lane (g, li) loads row 16 I + li, columns
//     32 p + 4 g .. + 3 and 32 p + 16 + 4 g .. + 3 (two 8-byte pieces).  The
//     next slot's tile is loaded while the current one is multiplied.
//   * P_{K-1} = A_{K-1} I is one pass with an identity B operand (exact).
//   * Per slot, before the multiply overwrites P_{j+1} in place: the affine
//     update (each lane's 16 products of its A pieces with c_{j+1}, summed
//     over the four lane groups), the apply (each lane's P values times
//     lambda_K, summed over the column blocks in the lane, then over the 16
//     lanes of a row), and the hi/lo split of P_{j+1}.
//   * c_j sits in a wave-private LDS ring of two vectors.
//
// All HIP code here is built with packed fp32 math disabled.

#include "lbi_device.hpp"
#include "lbi_internal.h"

namespace lbi {
namespace {

template <int R, bool AFF>
__global__ __launch_bounds__(64) void scan_wave_kernel(const ScanArgs args)
{
    constexpr int NB = R / 16;         // row and column blocks
    constexpr int NKP = (NB + 1) / 2;  // k pairs of the product
    constexpr int TILE = R * R * 2;    // bytes of one bf16 tile
    constexpr int VV = 4 * NB;         // apply values per lane before the row sums
    constexpr int VFF = VV >= 16 ? VV / 16 : 1;
    constexpr int SH = VV >= 16 ? 0 : (VV == 8 ? 1 : 2);
    __shared__ __attribute__((aligned(16))) float sc[AFF ? 2 : 1][AFF ? R : 4];

    const int lane = threadIdx.x;
    const int g = lane >> 4, li = lane & 15;
    const int64_t beta = blockIdx.x;
    const int64_t K = args.K;
    const __bf16 *A = (const __bf16 *)args.A + beta * K * (int64_t)(R * R);
    const __bf16 *bv = AFF ? (const __bf16 *)args.b + beta * K * (int64_t)R : nullptr;
    float *lam = args.lam + beta * K * (int64_t)R;
    auto ring = [&](int64_t s) { return (int)((K - 1 - s) & 1); };

    // ---- loads (branch-free: a slot outside the chain reads zeros) ----------
    // areg[set][I][p][piece]; breg[set]: b_j at row 16 g + li (raw bits << 16)
    u2 areg[2][NB][NKP][2];
    uint32_t breg[2];
    auto load_slot = [&](u2 (&dst)[NB][NKP][2], uint32_t &bdst, int64_t j) {
        const bool valid = j >= 0;
        const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
            (void *)(A + (valid ? j : 0) * (int64_t)(R * R)), 0, TILE, kBufferWord3);
#pragma unroll
        for (int I = 0; I < NB; ++I)
#pragma unroll
            for (int p = 0; p < NKP; ++p)
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const int col = 32 * p + 16 * h + 4 * g;
                    const int off = valid && col < R ? ((16 * I + li) * R + col) * 2 : kOutOfRange;
                    dst[I][p][h] = __builtin_amdgcn_raw_buffer_load_b64(rs, off, 0, 0);
                }
        if constexpr (AFF) {
            const __amdgpu_buffer_rsrc_t rb = __builtin_amdgcn_make_buffer_rsrc(
                (void *)(bv + (valid ? j : 0) * (int64_t)R), 0, R * 2, kBufferWord3);
            const int off = valid && g < NB ? (16 * g + li) * 2 : kOutOfRange;
            bdst = (uint32_t)__builtin_amdgcn_raw_buffer_load_b16(rb, off, 0, 0) << 16;
        }
    };
    auto a_op = [&](const u2 (&src)[NB][NKP][2], int I, int p) {
        return __builtin_bit_cast(bf16x8, u4{src[I][p][0][0], src[I][p][0][1],
                                             src[I][p][1][0], src[I][p][1][1]});
    };

    // lambda_K at the columns this lane multiplies
    float lk[NB];
#pragma unroll
    for (int cb = 0; cb < NB; ++cb)
        lk[cb] = (float)((const __bf16 *)args.lamK)[beta * R + 16 * cb + li];

    f4 P[NB][NB];  // [I][cb]

    // ---- lambda_s = P_s lambda_K + c_s, stored --------------------------------
    auto apply = [&](int64_t s) {
        float q[VV];
#pragma unroll
        for (int I = 0; I < NB; ++I)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                float t = P[I][0][v] * lk[0];
#pragma unroll
                for (int cb = 1; cb < NB; ++cb)
                    t += P[I][cb][v] * lk[cb];
                q[4 * I + v] = t;
            }
        group_reduce<16, VV>(q, li);
        const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
            (void *)(lam + s * (int64_t)R), 0, R * 4, kBufferWord3);
        const bool mine = (li & ((1 << SH) - 1)) == 0;
#pragma unroll
        for (int e = 0; e < VFF; ++e) {
            const int idx = (li >> SH) * VFF + e;  // = 4 I + v
            const int row = 16 * (idx >> 2) + 4 * g + (idx & 3);
            float val = q[e];
            if constexpr (AFF)
                val += sc[ring(s)][row];
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(val), rs,
                                                  mine ? row * 4 : kOutOfRange, 0, 0);
        }
    };

    // ---- slot K-1: P = A_{K-1} (identity B operand), c = b_{K-1} --------------
    load_slot(areg[0], breg[0], K - 1);
    load_slot(areg[1], breg[1], K - 2);
    {
        const __bf16 one = (__bf16)1.0f, zero = (__bf16)0.0f;
#pragma unroll
        for (int I = 0; I < NB; ++I)
#pragma unroll
            for (int cb = 0; cb < NB; ++cb)
                P[I][cb] = f4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int p = 0; p < NKP; ++p)
#pragma unroll
            for (int cb = 0; cb < NB; ++cb) {
                bf16x8 id;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const int k = 32 * p + (e < 4 ? 0 : 16) + 4 * g + (e & 3);
                    id[e] = k == 16 * cb + li ? one : zero;
                }
#pragma unroll
                for (int I = 0; I < NB; ++I)
                    P[I][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a_op(areg[0], I, p), id,
                                                                       P[I][cb], 0, 0, 0);
            }
        if constexpr (AFF) {
            if (g < NB)
                sc[ring(K - 1)][16 * g + li] = bitsf(breg[0]);
        }
    }
    load_slot(areg[0], breg[0], K - 3);

    // ---- slots K-2 .. 0 ---------------------------------------------------------
    // Slot j sits in register set (K-1-j) mod 2; after its product the set is
    // refilled with slot j-2.
    for (int64_t base = K - 2; base >= 0; base -= 2) {
#pragma unroll
        for (int s = 0; s < 2; ++s) {
            const int64_t j = base - s;
            if (j < 0)
                break;
            const int cur = (s + 1) & 1;  // (K-1-j) mod 2
            u2 (&aj)[NB][NKP][2] = cur ? areg[1] : areg[0];
            uint32_t &bj = cur ? breg[1] : breg[0];

            // c_j = A_j c_{j+1} + b_j
            if constexpr (AFF) {
                float part[NB];
#pragma unroll
                for (int I = 0; I < NB; ++I)
                    part[I] = 0.0f;
#pragma unroll
                for (int p = 0; p < NKP; ++p)
#pragma unroll
                    for (int h = 0; h < 2; ++h) {
                        const int col = 32 * p + 16 * h + 4 * g;
                        if (col < R) {
                            const f4 cv = *(const f4 *)&sc[ring(j + 1)][col];
#pragma unroll
                            for (int I = 0; I < NB; ++I) {
                                const u2 w = aj[I][p][h];
                                part[I] += bitsf(w[0] << 16) * cv[0] + bitsf(w[0] & kHighHalf) * cv[1] +
                                           bitsf(w[1] << 16) * cv[2] + bitsf(w[1] & kHighHalf) * cv[3];
                            }
                        }
                    }
                // every lane group holds a quarter of each row's k range: sum
                // over the four groups, then lane (g, li) keeps row 16 g + li
                float mine = 0.0f;
#pragma unroll
                for (int I = 0; I < NB; ++I) {
                    part[I] += __shfl_xor(part[I], 16);
                    part[I] += __shfl_xor(part[I], 32);
                    if (g == I)
                        mine = part[I];
                }
                __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
                __builtin_amdgcn_wave_barrier();
                __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
                if (g < NB)
                    sc[ring(j)][16 * g + li] = mine + bitsf(bj);
            }

            // lambda_{j+1} from P_{j+1}
            apply(j + 1);

            // P_j = A_j (P_{j+1} as bf16 hi + lo), in place
            bf16x8 bh[NKP][NB], bl[NKP][NB];
#pragma unroll
            for (int p = 0; p < NKP; ++p)
#pragma unroll
                for (int cb = 0; cb < NB; ++cb) {
                    u4 hh, ll;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        // values 2e, 2e+1 of the operand: rows 4 g + 2e.. of
                        // block 2p (e < 2) or of block 2p + 1 (e >= 2)
                        const int blk = 2 * p + (e >> 1);
                        const float x0 = blk < NB ? P[blk < NB ? blk : 0][cb][2 * (e & 1)] : 0.0f;
                        const float x1 = blk < NB ? P[blk < NB ? blk : 0][cb][2 * (e & 1) + 1] : 0.0f;
                        const uint32_t hu = __builtin_bit_cast(
                            uint32_t, __builtin_convertvector(f2{x0, x1}, bf16x2));
                        const f2 rest = {x0 - bitsf(hu << 16), x1 - bitsf(hu & kHighHalf)};
                        hh[e] = hu;
                        ll[e] = __builtin_bit_cast(uint32_t, __builtin_convertvector(rest, bf16x2));
                    }
                    bh[p][cb] = __builtin_bit_cast(bf16x8, hh);
                    bl[p][cb] = __builtin_bit_cast(bf16x8, ll);
                }
#pragma unroll
            for (int p = 0; p < NKP; ++p)
#pragma unroll
                for (int hl = 0; hl < 2; ++hl)
#pragma unroll
                    for (int I = 0; I < NB; ++I) {
                        const bf16x8 a = a_op(aj, I, p);
#pragma unroll
                        for (int cb = 0; cb < NB; ++cb) {
                            const f4 acc = p == 0 && hl == 0 ? f4{0.0f, 0.0f, 0.0f, 0.0f} : P[I][cb];
                            P[I][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                a, hl ? bl[p][cb] : bh[p][cb], acc, 0, 0, 0);
                        }
                    }
            load_slot(aj, bj, j - 2);
        }
    }
    apply(0);
}

template <int R>
hipError_t launch_r(const ChainLaunch &c)
{
    void *params[] = {(void *)&c.args};
    const void *fn = c.aff ? (const void *)&scan_wave_kernel<R, true>
                           : (const void *)&scan_wave_kernel<R, false>;
    return hipLaunchKernel(fn, dim3((unsigned)c.B), dim3(64), params, 0, c.stream);
}

}  // namespace

bool chain_wave_supported(const ChainLaunch &c)
{
    return c.out == kOutLambda && !c.args.progress && !c.args.compact && c.args.S == 1 &&
           (c.r == 16 || c.r == 32 || c.r == 64);
}

hipError_t launch_chain_wave_bf16(const ChainLaunch &c)
{
    if (!chain_wave_supported(c))
        return hipErrorInvalidValue;
    switch (c.r) {
    case 16: return launch_r<16>(c);
    case 32: return launch_r<32>(c);
    default: return launch_r<64>(c);
    }
}

}  // namespace lbi
