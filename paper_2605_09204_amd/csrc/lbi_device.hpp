// Device helpers shared by the kernels of the LBI scan library: vector
// types, lane exchanges within a wavefront, group reductions and the exact
// three-part bf16 split of fp32 values.
#ifndef LBI_DEVICE_HPP
#define LBI_DEVICE_HPP

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lbi {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef unsigned int u4 __attribute__((ext_vector_type(4)));
typedef unsigned int u2 __attribute__((ext_vector_type(2)));
typedef float f2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int waves_for(int R) { return R == 16 ? 1 : (R == 32 ? 2 : 4); }
constexpr int ilog2(int x) { return x <= 1 ? 0 : 1 + ilog2(x / 2); }

// Buffer resource word 3 for raw (untyped) buffer loads on gfx9-family GPUs.
constexpr int kBufferWord3 = 0x00020000;
// A per-lane offset past every tile: the load returns zero, no memory access.
constexpr int kOutOfRange = 0x40000000;
constexpr uint32_t kHighHalf = 0xFFFF0000u;

__device__ __forceinline__ int pow2_at_least(int x)
{
    return x <= 1 ? 1 : (x <= 2 ? 2 : (x <= 4 ? 4 : 8));
}

// DPP lane permutations within a 16-lane row (GFX9 encodings).
constexpr int kDppXor1 = 0xB1;   // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;   // quad_perm [2,3,0,1]
constexpr int kDppXor7 = 0x141;  // row_half_mirror: lane i <- i ^ 7
constexpr int kDppXor8 = 0x128;  // row_ror:8:       lane i <- i ^ 8

// (bound_ctrl set, all rows and banks enabled: the compiler can fold the move
// into the instruction that consumes it)
template <int CTRL> __device__ __forceinline__ float dpp(float x)
{
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), CTRL, 0xF, 0xF, true));
}

// The value of lane (this lane ^ MASK); MASK 7 stands in for 4 (it flips the
// same top bit of an 8-lane group, and together with 2 and 1 it still spans
// every lane of the group).
template <int MASK> __device__ __forceinline__ float xchg(float x)
{
    if constexpr (MASK == 1) return dpp<kDppXor1>(x);
    else if constexpr (MASK == 2) return dpp<kDppXor2>(x);
    else if constexpr (MASK == 7) return dpp<kDppXor7>(x);
    else if constexpr (MASK == 8) return dpp<kDppXor8>(x);
    else {
        static_assert(MASK == 16, "lane exchange");
        return __shfl_xor(x, 16);
    }
}

// One halving stage for the partner masks 8 and 7, without selects: DPP's
// bank mask (the 4-lane banks of a 16-lane row) limits which lanes write.
// Lanes whose stage bit is 0 fill banks LO, the others banks HI (bit 3 of the
// lane: banks 0-1 / 2-3; bit 2: banks 0, 2 / 1, 3).  For each pair
// (a, b) = (q[i], b[i]): a <- a + partner's a in the LO lanes, then
// a <- b + partner's b in the HI lanes; neither step reads what the other
// writes.  A DPP read needs two wait states after a VALU write of the same
// register, and the compiler does not see the writes inside an asm block, so
// each block starts and ends with s_nop 1.
#define LBI_HALF_PAIR(CTRL, LO, HI, A, B)                                                    \
    "v_add_f32_dpp %" #A ", %" #A ", %" #A " " CTRL " row_mask:0xf bank_mask:" LO "\n\t" \
    "v_add_f32_dpp %" #A ", %" #B ", %" #B " " CTRL " row_mask:0xf bank_mask:" HI "\n\t"
#define LBI_HB8(C, L, U) LBI_HALF_PAIR(C, L, U, 0, 8) LBI_HALF_PAIR(C, L, U, 1, 9)             \
    LBI_HALF_PAIR(C, L, U, 2, 10) LBI_HALF_PAIR(C, L, U, 3, 11) LBI_HALF_PAIR(C, L, U, 4, 12) \
    LBI_HALF_PAIR(C, L, U, 5, 13) LBI_HALF_PAIR(C, L, U, 6, 14) LBI_HALF_PAIR(C, L, U, 7, 15)
#define LBI_HB4(C, L, U) LBI_HALF_PAIR(C, L, U, 0, 4) LBI_HALF_PAIR(C, L, U, 1, 5)             \
    LBI_HALF_PAIR(C, L, U, 2, 6) LBI_HALF_PAIR(C, L, U, 3, 7)
#define LBI_HB2(C, L, U) LBI_HALF_PAIR(C, L, U, 0, 2) LBI_HALF_PAIR(C, L, U, 1, 3)
#define LBI_HB1(C, L, U) LBI_HALF_PAIR(C, L, U, 0, 1)
#define LBI_HB(PAIRS)                                                                         \
    if constexpr (MASK == 8)                                                                  \
        asm("s_nop 1\n\t" PAIRS("row_ror:8", "0x3", "0xc") "s_nop 1" : LBI_HB_OPS);          \
    else                                                                                      \
        asm("s_nop 1\n\t" PAIRS("row_half_mirror", "0x5", "0xa") "s_nop 1" : LBI_HB_OPS);
template <int MASK, int H> __device__ __forceinline__ void halve_banked(float *q, const float *b)
{
    static_assert(MASK == 8 || MASK == 7, "bank-masked halving");
    if constexpr (H == 8) {
#define LBI_HB_OPS "+v"(q[0]), "+v"(q[1]), "+v"(q[2]), "+v"(q[3]), "+v"(q[4]), "+v"(q[5]), \
                   "+v"(q[6]), "+v"(q[7]) : "v"(b[0]), "v"(b[1]), "v"(b[2]), "v"(b[3]),   \
                   "v"(b[4]), "v"(b[5]), "v"(b[6]), "v"(b[7])
        LBI_HB(LBI_HB8)
#undef LBI_HB_OPS
    } else if constexpr (H == 4) {
#define LBI_HB_OPS "+v"(q[0]), "+v"(q[1]), "+v"(q[2]), "+v"(q[3]) : "v"(b[0]), "v"(b[1]), "v"(b[2]), "v"(b[3])
        LBI_HB(LBI_HB4)
#undef LBI_HB_OPS
    } else if constexpr (H == 2) {
#define LBI_HB_OPS "+v"(q[0]), "+v"(q[1]) : "v"(b[0]), "v"(b[1])
        LBI_HB(LBI_HB2)
#undef LBI_HB_OPS
    } else {
        static_assert(H == 1, "pairs per stage");
#define LBI_HB_OPS "+v"(q[0]) : "v"(b[0])
        LBI_HB(LBI_HB1)
#undef LBI_HB_OPS
    }
}
#undef LBI_HB
#undef LBI_HB1
#undef LBI_HB2
#undef LBI_HB4
#undef LBI_HB8
#undef LBI_HALF_PAIR

// Sum LIVE values per lane over an aligned group of N lanes (gi = lane index
// in the group, which is also the lane's index modulo N: the masks 8 and 7
// go by hardware lane position).  Each stage either halves the live values
// (lanes whose bit BIT is 0 keep the lower half, summed with the partner's
// lower half, the others the upper) or, with one value left, adds the
// partner's.  Afterwards lane gi holds, in q[e] for e < max(1, LIVE / N), the
// full group sum of original index (gi >> S) * max(1, LIVE / N) + e with
// S = log2(N) - log2(min(LIVE, N)).
template <int N, int LIVE, int V> __device__ __forceinline__ void group_reduce(float (&q)[V], int gi)
{
    if constexpr (N > 1) {
        constexpr int MASK = N == 32 ? 16 : (N == 16 ? 8 : (N == 8 ? 7 : (N == 4 ? 2 : 1)));
        constexpr int BIT = ilog2(N) - 1;
        if constexpr (LIVE >= 2 && (MASK == 8 || MASK == 7)) {
#pragma unroll
            for (int i = 0; i < LIVE / 2; i += 8)
                halve_banked<MASK, (LIVE / 2 < 8 ? LIVE / 2 : 8)>(q + i, q + i + LIVE / 2);
            group_reduce<N / 2, LIVE / 2>(q, gi);
        } else if constexpr (LIVE >= 2) {
            const bool upper = (gi >> BIT) & 1;
#pragma unroll
            for (int i = 0; i < LIVE / 2; ++i) {
                const float keep = upper ? q[i + LIVE / 2] : q[i];
                const float send = upper ? q[i] : q[i + LIVE / 2];
                q[i] = keep + xchg<MASK>(send);
            }
            group_reduce<N / 2, LIVE / 2>(q, gi);
        } else {
            q[0] += xchg<MASK>(q[0]);
            group_reduce<N / 2, 1>(q, gi);
        }
    }
}

template <typename T> __device__ __forceinline__ float to_f32(T x) { return (float)x; }

__device__ __forceinline__ uint32_t fbits(float x) { return __float_as_uint(x); }
__device__ __forceinline__ float bitsf(uint32_t u) { return __uint_as_float(u); }

// Three bf16 parts of two fp32 values with h + m + l == x exactly (for
// normal x), each packed as the bf16 pair (part of x0, part of x1):
//   h = x rounded to the nearest bf16; the remainder r = x - h is exact and
//       has at most 16 significant bits (|r| <= half an ulp of h);
//   m = r rounded to the nearest bf16; l = r - m is exact and has at most 8
//       significant bits, so it is a bf16 value.
// Rounding to nearest, rather than truncating, keeps every part centred: the
// partial products that the six-product scheme leaves out then have no sign
// bias, and their rounding does not build up along a long chain of products.
// Each remainder is one bf16 dot product, x - 1 * part, which is exact.  The
// selectors (-1, 0) and (0, -1) are passed in registers: an inline constant
// in a packed bf16 operand is not read as a bf16 pair.
struct Split2 {
    uint32_t h, m, l;
};
__device__ __forceinline__ Split2 split_pair(float x0, float x1)
{
    uint32_t sel0 = 0x0000BF80u, sel1 = 0xBF800000u;  // bf16 pairs (-1, 0), (0, -1)
    asm("" : "+v"(sel0), "+v"(sel1));
    const bf16x2 neg0 = __builtin_bit_cast(bf16x2, sel0);
    const bf16x2 neg1 = __builtin_bit_cast(bf16x2, sel1);
    const bf16x2 h = __builtin_convertvector(f2{x0, x1}, bf16x2);
    const float r0 = __builtin_amdgcn_fdot2_f32_bf16(h, neg0, x0, false);
    const float r1 = __builtin_amdgcn_fdot2_f32_bf16(h, neg1, x1, false);
    const bf16x2 m = __builtin_convertvector(f2{r0, r1}, bf16x2);
    const float l0 = __builtin_amdgcn_fdot2_f32_bf16(m, neg0, r0, false);
    const float l1 = __builtin_amdgcn_fdot2_f32_bf16(m, neg1, r1, false);
    const bf16x2 l = __builtin_convertvector(f2{l0, l1}, bf16x2);
    return {__builtin_bit_cast(uint32_t, h), __builtin_bit_cast(uint32_t, m),
            __builtin_bit_cast(uint32_t, l)};
}

// The same three parts, with each remainder formed as x - part by an fp32
// subtraction (exact for the same reason), which leaves x in its register:
// for values that are still needed after the split.  (The dot-product form
// above accumulates into its third operand, so the compiler copies x first
// when x stays live.)
__device__ __forceinline__ Split2 split_pair_keep(float x0, float x1)
{
    const uint32_t h = __builtin_bit_cast(uint32_t, __builtin_convertvector(f2{x0, x1}, bf16x2));
    const float r0 = x0 - bitsf(h << 16), r1 = x1 - bitsf(h & kHighHalf);
    const uint32_t m = __builtin_bit_cast(uint32_t, __builtin_convertvector(f2{r0, r1}, bf16x2));
    const float l0 = r0 - bitsf(m << 16), l1 = r1 - bitsf(m & kHighHalf);
    const uint32_t l = __builtin_bit_cast(uint32_t, __builtin_convertvector(f2{l0, l1}, bf16x2));
    return {h, m, l};
}

}  // namespace
}  // namespace lbi

#endif  // LBI_DEVICE_HPP
