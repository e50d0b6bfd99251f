// The log-depth (tree) scan of the LBI interface-adjoint recurrence on gfx950.
//
// Proposition "Scan Formulation of Backpropagation" lets the suffix products
// be formed by any associative scan; its span term in Proposition
// "Work-Span Decomposition" is logarithmic in K.  This file builds that
// scan as a Blelloch tree with a matrix up-sweep and a vector down-sweep:
//
//   up-sweep   node(i, 2s) = node(i, s) o node(i + s, s) for i = 0, 2s, 4s,
//              ... (the combine (P, c) o (P', c') = (P P', P c' + c), left
//              operand the lower slots), s = 1, 2, 4, ...: K - 1 matrix
//              products in all (as many as a right-to-left fold), log2 of the
//              chunk in depth;
//   down-sweep lambda at the lower end of a node from lambda at its upper end,
//              lambda_i = P lambda_{i + s} + c: the vector form of the
//              down-sweep (only adjoints are needed, never the prefix
//              matrices), again logarithmic in depth.
//
// One workgroup takes a chunk of C consecutive slots of one chain (C = 8 at
// r = 64, 16 below) and keeps every node as an fp32 tile in LDS.  A node
// is written over the tile of its left child, so the tile of slot w ends up
// holding node(w, lowbit(w)) (node(0, C) for w = 0), which is exactly the
// right child that the down-sweep needs at w: lambda_w = node(w, lowbit(w))
// lambda_{w + lowbit(w)}.  Going down by decreasing lowbit, every lambda it
// reads was formed in an earlier step, and there are log2(C) steps.
//
// The matrix products run on the bf16 matrix cores in the exact three-part
// split of the chain scan (every fp32 operand cut into three bf16 parts whose
// sum is the value; the six partial products down to 2^-16 of the leading
// one, fp32 accumulation).  A level's products are cut into units of one
// product and one to four 16-column blocks, one unit per wave, so that all
// waves work while there are enough products; the affine parts P c' + c are
// matrix-vector products (one lane per row) in further units.  Each wave
// keeps its unit's result in registers until a barrier says every operand
// has been read, then writes it over the left child.
//
// Chains longer than C are scanned over levels: a pass of this kernel writes
// each chunk's aggregate (its node(0, n)), the aggregates form a chain C
// times shorter, and so on until one chunk remains; that chunk is scanned to
// lambda from lambda_K, and then each level is scanned again from the lambda
// at the start of the next chunk (its carry).  2L + 1 launches for
// K <= C^(L+1).
//
// All HIP code here is built with packed fp32 math disabled.

#include "lbi_device.hpp"
#include "lbi_internal.h"

namespace lbi {
namespace {

template <int R> struct TreeGeo {
    static constexpr int C = R == 64 ? 8 : 16;     // slots per chunk
    static constexpr int LOGC = R == 64 ? 3 : 4;
    static constexpr int NW = C;                    // waves per workgroup
    static constexpr int T = 64 * NW;
    static constexpr int PITCH = R + 4;             // fp32 row pitch of an LDS tile
    static constexpr int TILE = R * PITCH;
    static constexpr int NB = R / 16;               // 16-row (and -column) blocks
    static constexpr int NKP = R >= 32 ? R / 32 : 1;  // k pairs of 32 (r = 16: one, half zero)
};

// Column blocks per unit at a level with at most `ncomb` products.  Every
// unit splits all of its left operand (and its own columns of the right
// one) into bf16 parts, and that VALU work, not the matrix cores, sets a
// level's time: so a level gets about NB units in all, one per SIMD at
// r = 64, each as wide as that allows (at r = 64, C = 8 the three levels
// take 4 units of 4, 4 units of 2 and 4 units of 1 column block: measured
// 7.5k, 4.9k and 3.5k cycles, against 9.5k, 6.8k and 3.5k with one unit
// per wave).
template <int R> constexpr int cb_per_unit(int ncomb)
{
    using G = TreeGeo<R>;
    int u = G::NB / ncomb;  // units per product
    if (u < 1)
        u = 1;
    return G::NB / u;
}

// Eight consecutive k values of the B operand (rows 32p + 4g + e and
// 32p + 16 + 4g + e of column col of an fp32 LDS tile), split into three bf16
// planes.  r = 16 has one k block of 16: the upper half is zero.
template <int R>
__device__ __forceinline__ void b_split(const float *tile, int p, int g, int col, bf16x8 &h,
                                        bf16x8 &m, bf16x8 &l)
{
    using G = TreeGeo<R>;
    float x[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        x[e] = tile[(32 * p + 4 * g + e) * G::PITCH + col];
        x[e + 4] = R >= 32 ? tile[(32 * p + 16 + 4 * g + e) * G::PITCH + col] : 0.0f;
    }
    u4 hh, mm, ll;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const Split2 s = split_pair(x[2 * e], x[2 * e + 1]);
        hh[e] = s.h;
        mm[e] = s.m;
        ll[e] = s.l;
    }
    h = __builtin_bit_cast(bf16x8, hh);
    m = __builtin_bit_cast(bf16x8, mm);
    l = __builtin_bit_cast(bf16x8, ll);
}

// The same eight k values of row `row` as the A operand (two 16-byte reads).
template <int R>
__device__ __forceinline__ void a_split(const float *tile, int p, int g, int row, bf16x8 &h,
                                        bf16x8 &m, bf16x8 &l)
{
    using G = TreeGeo<R>;
    const f4 lo = *(const f4 *)&tile[row * G::PITCH + 32 * p + 4 * g];
    const f4 hi = R >= 32 ? *(const f4 *)&tile[row * G::PITCH + 32 * p + 16 + 4 * g]
                          : f4{0.0f, 0.0f, 0.0f, 0.0f};
    const Split2 s0 = split_pair(lo[0], lo[1]), s1 = split_pair(lo[2], lo[3]);
    const Split2 s2 = split_pair(hi[0], hi[1]), s3 = split_pair(hi[2], hi[3]);
    h = __builtin_bit_cast(bf16x8, u4{s0.h, s1.h, s2.h, s3.h});
    m = __builtin_bit_cast(bf16x8, u4{s0.m, s1.m, s2.m, s3.m});
    l = __builtin_bit_cast(bf16x8, u4{s0.l, s1.l, s2.l, s3.l});
}

// acc = PL * PR[:, column blocks cb0 .. cb0 + CBU - 1], in the accumulator
// layout (lane (g, li) of block (I, t) holds rows 16 I + 4 g + v, column
// 16 (cb0 + t) + li).  Both operands fp32 tiles in LDS.  EXACT: both are
// bf16 values held in fp32 (the leaves of a bf16 chain), so the leading
// parts are the values and one product is exact.
template <int R, int CBU, bool EXACT>
__device__ __forceinline__ void product_unit(const float *PL, const float *PR, int cb0, int g,
                                             int li, f4 (&acc)[TreeGeo<R>::NB][CBU])
{
    using G = TreeGeo<R>;
#pragma unroll
    for (int I = 0; I < G::NB; ++I)
#pragma unroll
        for (int t = 0; t < CBU; ++t)
            acc[I][t] = f4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int p = 0; p < G::NKP; ++p) {
        bf16x8 bh[CBU], bm[CBU], bl[CBU];
#pragma unroll
        for (int t = 0; t < CBU; ++t)
            b_split<R>(PR, p, g, 16 * (cb0 + t) + li, bh[t], bm[t], bl[t]);
#pragma unroll
        for (int I = 0; I < G::NB; ++I) {
            bf16x8 ah, am, al;
            a_split<R>(PL, p, g, 16 * I + li, ah, am, al);
#pragma unroll
            for (int t = 0; t < CBU; ++t) {
                f4 c = acc[I][t];
                c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bh[t], c, 0, 0, 0);
                if constexpr (EXACT) {
                    acc[I][t] = c;
                    continue;
                }
                c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bm[t], c, 0, 0, 0);
                c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(am, bh[t], c, 0, 0, 0);
                c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bl[t], c, 0, 0, 0);
                c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, bh[t], c, 0, 0, 0);
                c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(am, bm[t], c, 0, 0, 0);
                acc[I][t] = c;
            }
        }
    }
}

// y = P x (+ c) for one row per lane (lanes past R give 0): P an fp32 LDS
// tile, x and c LDS vectors (c may be NULL).
template <int R>
__device__ __forceinline__ float row_matvec(const float *P, const float *x, const float *c,
                                            int row)
{
    using G = TreeGeo<R>;
    if (row >= R)
        return 0.0f;
    float acc = 0.0f;
#pragma unroll
    for (int k = 0; k < R; k += 4) {
        const f4 p = *(const f4 *)&P[row * G::PITCH + k];
        const f4 v = *(const f4 *)&x[k];
        acc = fmaf(p[0], v[0], acc);
        acc = fmaf(p[1], v[1], acc);
        acc = fmaf(p[2], v[2], acc);
        acc = fmaf(p[3], v[3], acc);
    }
    return c ? acc + c[row] : acc;
}

// One level of the up-sweep: for every i = 0, 2s, 4s, ... with i + s < n,
// node(i) <- node(i) o node(i + s).  Product units first (NCOMB products of
// NB / CBU units each), then (affine) one matrix-vector unit per product.
template <int R, bool AFF, int LEV, bool LEAF_BF16>
__device__ __forceinline__ void up_level(float *sT, float (*sC)[R], int n, int w, int g, int li,
                                         int lane)
{
    using G = TreeGeo<R>;
    constexpr int s = 1 << (LEV - 1);
    constexpr int NCOMB = G::C >> LEV;  // products at this level in a full chunk
    constexpr int CBU = cb_per_unit<R>(NCOMB);
    constexpr int UPC = G::NB / CBU;    // product units per product
    const int ncomb = n > s ? (n - s + 2 * s - 1) / (2 * s) : 0;
    // this wave's product unit (at most one: NCOMB * UPC <= NW, counted from
    // wave 0) and matrix-vector unit (at most one, counted from the last
    // wave: a wave may hold one of each)
    static_assert(NCOMB * UPC <= G::NW && NCOMB <= G::NW, "units per level");
    const int pu = w;
    const bool has_p = pu < ncomb * UPC;
    const int pi = has_p ? (pu / UPC) * 2 * s : 0;
    const int cb0 = (pu % UPC) * CBU;
    const int mu = G::NW - 1 - w;
    const bool has_m = AFF && mu < ncomb;
    const int mi = has_m ? mu * 2 * s : 0;
    f4 acc[G::NB][CBU];
    float cnew = 0.0f;
    if (has_p)
        product_unit<R, CBU, LEV == 1 && LEAF_BF16>(sT + pi * G::TILE, sT + (pi + s) * G::TILE,
                                                    cb0, g, li, acc);
    if constexpr (AFF) {
        if (has_m)
            cnew = row_matvec<R>(sT + mi * G::TILE, sC[mi + s], sC[mi], lane);
    }
    __syncthreads();  // every operand of this level has been read
    if (has_p) {
        float *PL = sT + pi * G::TILE;
#pragma unroll
        for (int I = 0; I < G::NB; ++I)
#pragma unroll
            for (int t = 0; t < CBU; ++t)
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    PL[(16 * I + 4 * g + v) * G::PITCH + 16 * (cb0 + t) + li] = acc[I][t][v];
    }
    if constexpr (AFF) {
        if (has_m && lane < R)
            sC[mi][lane] = cnew;
    }
    __syncthreads();
}

// One chunk of C slots of one chain: the up-sweep, then either the chunk's
// aggregate (AGG) or every lambda of the chunk from its carry.
//   E: storage of A and b (float or bf16); the carry lambda_K is bf16 or fp32
//   by a.lamK_bf16; the carries of the level above (lamNext) are fp32.
template <int R, typename E, bool AFF, bool AGG>
__global__ __launch_bounds__(64 * TreeGeo<R>::NW) void scan_tree_kernel(const TreeArgs a)
{
    using G = TreeGeo<R>;
    __shared__ __attribute__((aligned(16))) float sT[G::C * G::TILE];
    __shared__ __attribute__((aligned(16))) float sC[AFF ? G::C : 1][R];
    __shared__ __attribute__((aligned(16))) float sL[AGG ? 1 : G::C + 1][R];

    const int tid = (int)threadIdx.x;
    const int lane = tid & 63, w = tid >> 6, g = lane >> 4, li = lane & 15;
    const int64_t beta = blockIdx.x / a.S;
    const int d = (int)(blockIdx.x % a.S);
    const int64_t s0 = (int64_t)d * G::C;
    const int n = (int)(a.K - s0 < G::C ? a.K - s0 : G::C);
    const int64_t first = beta * a.K + s0;  // global slot index of local slot 0

    // ---- the chunk's tiles and affine terms into LDS (fp32) -------------------
    {
        // The chunk's n tiles are one contiguous run of n R^2 elements: group
        // q of four elements (slot q / Q, row, column 4 c4) sits at element
        // 4 q.  Every load is issued before any LDS store (branch-free: groups
        // past the run get an out-of-range offset, which returns zeros
        // without a memory access), then the stores.
        constexpr int Q = R * R / 4;                  // groups per tile
        constexpr int NL = G::C * Q / G::T;           // groups per thread
        static_assert(NL * G::T == G::C * Q, "load geometry");
        const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
            (void *)((const E *)a.A + first * (int64_t)(R * R)), 0,
            n * R * R * (int)sizeof(E), kBufferWord3);
        f4 v[NL];
#pragma unroll
        for (int i = 0; i < NL; ++i) {
            const int q = i * G::T + tid;
            const int off = q < n * Q ? q * 4 * (int)sizeof(E) : kOutOfRange;
            if constexpr (sizeof(E) == 4) {
                v[i] = __builtin_bit_cast(f4, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0));
            } else {
                const u2 u = __builtin_amdgcn_raw_buffer_load_b64(rs, off, 0, 0);
                v[i] = f4{bitsf(u[0] << 16), bitsf(u[0] & kHighHalf), bitsf(u[1] << 16),
                          bitsf(u[1] & kHighHalf)};
            }
        }
#pragma unroll
        for (int i = 0; i < NL; ++i) {
            const int q = i * G::T + tid;
            const int slot = q / Q, within = q % Q;
            const int row = within / (R / 4), c4 = within % (R / 4);
            *(f4 *)&sT[slot * G::TILE + row * G::PITCH + 4 * c4] = v[i];
        }
        if constexpr (AFF) {
            const E *bv = (const E *)a.b + first * (int64_t)R;
            for (int q = tid; q < n * R; q += G::T)
                sC[q / R][q % R] = to_f32(bv[q]);
        }
        if constexpr (!AGG) {
            // lambda at the chunk's upper end: lambda_K for the last chunk,
            // else lambda at the start of the next chunk (the level above)
            if (tid < R) {
                float carry;
                if (d + 1 < a.S)
                    carry = a.lamNext[(beta * a.S + d + 1) * R + tid];
                else if (a.lamK_bf16)
                    carry = to_f32(((const __bf16 *)a.lamK)[beta * R + tid]);
                else
                    carry = ((const float *)a.lamK)[beta * R + tid];
                sL[n][tid] = carry;
            }
        }
    }
    __syncthreads();

    // ---- up-sweep: log2(C) levels --------------------------------------------
    constexpr bool LB = sizeof(E) == 2;
    up_level<R, AFF, 1, LB>(sT, sC, n, w, g, li, lane);
    up_level<R, AFF, 2, LB>(sT, sC, n, w, g, li, lane);
    up_level<R, AFF, 3, LB>(sT, sC, n, w, g, li, lane);
    if constexpr (G::LOGC >= 4)
        up_level<R, AFF, 4, LB>(sT, sC, n, w, g, li, lane);

    if constexpr (AGG) {
        // the chunk's aggregate node(0, n): tile 0 and its affine part
        float *P = a.Pagg + (beta * a.S + d) * (int64_t)(R * R);
        for (int q = tid; q < R * R / 4; q += G::T) {
            const int row = q / (R / 4), c4 = q % (R / 4);
            *(f4 *)&P[row * R + 4 * c4] = *(const f4 *)&sT[row * G::PITCH + 4 * c4];
        }
        if (a.cagg && tid < R)
            a.cagg[(beta * a.S + d) * R + tid] = AFF ? sC[0][tid] : 0.0f;
    } else {
        // ---- down-sweep: lambda_w = node(w, lowbit(w)) lambda_{e(w)} + c ------
        // (e(w) = min(w + lowbit(w), n), lowbit(0) = C); by decreasing lowbit
        float *lam = a.lam + first * (int64_t)R;
#pragma unroll
        for (int step = G::LOGC; step >= 1; --step) {
            const int low = 1 << (step - 1);  // lowbit of the slots of this step
            // slots w = low, 3 low, 5 low, ... (< n), and w = 0 in the first step
            const int nlow = n > low ? (n - low + 2 * low - 1) / (2 * low) : 0;
            const int extra = step == G::LOGC ? 1 : 0;
            if (w < nlow + extra) {
                const int slot = w < nlow ? (2 * w + 1) * low : 0;
                const int span = slot == 0 ? G::C : low;
                const int e = slot + span < n ? slot + span : n;
                const float y = row_matvec<R>(sT + slot * G::TILE, sL[e],
                                              AFF ? sC[AFF ? slot : 0] : nullptr, lane);
                if (lane < R) {
                    sL[slot][lane] = y;
                    lam[(int64_t)slot * R + lane] = y;
                }
            }
            __syncthreads();
        }
    }
}

template <int R, typename E, bool AFF, bool AGG>
hipError_t tree_launch(const TreeArgs &a, int64_t B, hipStream_t stream)
{
    void *params[] = {(void *)&a};
    return hipLaunchKernel((const void *)&scan_tree_kernel<R, E, AFF, AGG>,
                           dim3((unsigned)(B * a.S)), dim3(TreeGeo<R>::T), params, 0, stream);
}

template <int R, typename E>
hipError_t tree_dispatch(const TreeArgs &a, int64_t B, bool aff, bool agg, hipStream_t stream)
{
    if (agg)
        return aff ? tree_launch<R, E, true, true>(a, B, stream)
                   : tree_launch<R, E, false, true>(a, B, stream);
    return aff ? tree_launch<R, E, true, false>(a, B, stream)
               : tree_launch<R, E, false, false>(a, B, stream);
}

}  // namespace

int tree_chunk(int32_t r) { return r == 64 ? TreeGeo<64>::C : TreeGeo<32>::C; }

hipError_t launch_tree(const TreeArgs &a, int64_t B, int32_t r, bool a_bf16, bool aff, bool agg,
                       hipStream_t stream)
{
    switch (r) {
    case 16:
        return a_bf16 ? tree_dispatch<16, __bf16>(a, B, aff, agg, stream)
                      : tree_dispatch<16, float>(a, B, aff, agg, stream);
    case 32:
        return a_bf16 ? tree_dispatch<32, __bf16>(a, B, aff, agg, stream)
                      : tree_dispatch<32, float>(a, B, aff, agg, stream);
    case 64:
        return a_bf16 ? tree_dispatch<64, __bf16>(a, B, aff, agg, stream)
                      : tree_dispatch<64, float>(a, B, aff, agg, stream);
    default:
        return hipErrorInvalidValue;
    }
}

}  // namespace lbi
