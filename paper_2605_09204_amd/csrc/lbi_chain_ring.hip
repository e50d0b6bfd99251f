// The chain scan with the A_j tiles streamed into an LDS ring by direct
// HBM-to-LDS loads (bf16 storage; interface widths 32, 64 or 128, r_K = 64).
//
// Computes what the workgroup-per-chain kernel computes, for B independent
// chains of K slots: the suffix composites
//     (P_j, c_j) = (A_j, b_j) o (A_{j+1}, b_{j+1}) o ... o (A_{K-1}, b_{K-1})
// with the combine (A, b) o (A', b') = (A A', A b' + b) of the scan
// formulation (Proposition "Scan Formulation of Backpropagation"), and
// lambda_j = P_j lambda_K + c_j for every slot (Phase 2 of Algorithm
// "Bounded-Interface Backpropagation").  One workgroup of four waves folds one
// chain from its end.  The design trades the register staging of that kernel
// for hardware that gfx950 offers, so that four chains fit on a CU:
//   * Tiles go HBM -> LDS with `buffer_load_dwordx4 ... lds`: each lane's 16
//     bytes land at M0 + 16 * lane, no VGPRs and no VALU work in between.
//     A tile is cut into 1 KB blocks of 16 rows x 32 columns, one load
//     instruction per block.  Tiles j, j-1 and j-2 are resident at once
//     (prefetch two slots ahead), in a ring of blocks sized by the host for
//     the chain's widths: only the live r_j x r_{j+1} part of a zero-padded
//     tile is read, and slots of different shapes share the ring.
//   * The loads are issued from inline assembly, so the compiler does not
//     track them; each slot barrier waits for them with an explicit vector
//     memory count: the wave's operations issued since are the next tile's
//     loads (a number the widths fix) and two lambda stores.
//   * Row order: LDS row m of a tile holds tile row
//     sigma(m) = 32 (m / 32) + 8 ((m % 16) / 4) + 4 ((m / 16) % 2) + m % 4.
//     The running composite P sits in MFMA accumulator layout (lane l holds
//     rows 16 I + 4 (l / 16) + v of column 16 w + l % 16), which is also the
//     B-operand layout of the next product; with rows in sigma order the k
//     values a lane holds for 32-wide k block p are the true rows
//     32 p + 8 (l / 16) + 0..7, so the A operand is a natural 16-byte chunk
//     of the tile row.  Chunks within a block row are XOR-swizzled by
//     (row / 4) % 4, which puts the 16 lanes of an operand read on distinct
//     banks.
//   * P_j = A_j P_{j+1} on v_mfma_f32_16x16x32_bf16, the fp32 composite fed
//     back as bf16 hi + lo; wave w of NW owns column blocks w, w + NW, ....
//   * c_j = A_j c_{j+1} + b_j on the matrix cores as well: c_{j+1} (hi + lo,
//     the same value in all 16 columns of a B operand) against the A operands
//     already read for P, row block I by wave I % NW.  The wave then adds b_j
//     to its rows and writes c_j (fp32, for lambda) and its bf16 parts (the
//     next slot's operand) to LDS.
//   * lambda_j: per-wave partial P_{j+1} lambda_K (a DPP butterfly over the
//     16 lanes of a column block), summed across the waves through LDS with
//     c_j and stored once, coalesced, by a pair of waves.
//   * Waves per chain: four at storage width 64 (one column block each, at
//     most 128 VGPRs); two at width 128 (two column blocks each, up to 256
//     VGPRs), which halves the per-wave bookkeeping of a chain and measured
//     faster there.
//
// All HIP code here is built with packed fp32 math disabled.

#include "lbi_device.hpp"
#include "lbi_internal.h"

namespace lbi {
namespace {

typedef int i4 __attribute__((ext_vector_type(4)));

constexpr int kBlk = 1024;  // bytes of one 16-row x 32-column bf16 block

// Waves per chain by storage width (4: one composite column block each, 2:
// two each).
#ifndef LBI_RING_NW64
#define LBI_RING_NW64 4
#endif
#ifndef LBI_RING_NW128
#define LBI_RING_NW128 2
#endif

// Dynamic LDS layout (bytes) for a ring of `ring` blocks.
struct RingLds {
    int part, c, cop, b, total;
};
__host__ __device__ constexpr RingLds ring_lds(int ring, bool aff)
{
    RingLds o{};
    o.part = ring * kBlk;             // [2][4 waves][128] fp32 partial applies
    o.c = o.part + 2 * 4 * 128 * 4;   // [4][128] fp32 c_j, by true row
    o.cop = o.c + (aff ? 4 * 128 * 4 : 0);   // [2][hi, lo][128] bf16 c operand
    o.b = o.cop + (aff ? 2 * 2 * 128 * 2 : 0);  // [3][128] bf16 b_j
    o.total = o.b + (aff ? 3 * 128 * 2 : 0);
    return o;
}

// Tile row held by LDS row 16 I + li.
__device__ __forceinline__ int sigma_row(int I, int li)
{
    return 32 * (I >> 1) + 4 * (I & 1) + 8 * (li >> 2) + (li & 3);
}

__device__ __forceinline__ i4 rsrc(const void *base, uint32_t bytes)
{
    const uint64_t a = (uint64_t)(uintptr_t)base;
    i4 r;
    r[0] = (int)(uint32_t)a;
    r[1] = (int)((uint32_t)(a >> 32) & 0xFFFFu);
    r[2] = (int)bytes;
    r[3] = kBufferWord3;
    return r;
}

// 16 bytes per lane from rs at voff + soff into LDS at lds + 16 * lane; M0
// (the LDS destination, one wait state after writing it) is saved and
// restored inside the asm.
__device__ __forceinline__ void dma_b128(uint32_t lds, i4 rs, int voff, int soff)
{
    uint32_t keep;
    asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %1\n\ts_nop 0\n\t"
                 "buffer_load_dwordx4 %2, %3, %4 offen lds\n\ts_mov_b32 m0, %0"
                 : "=&s"(keep)
                 : "s"(lds), "v"(voff), "s"(rs), "s"(soff)
                 : "memory");
}
// 4 bytes per lane into LDS at lds + 4 * lane.
__device__ __forceinline__ void dma_b32(uint32_t lds, i4 rs, int voff, int soff)
{
    uint32_t keep;
    asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %1\n\ts_nop 0\n\t"
                 "buffer_load_dword %2, %3, %4 offen lds\n\ts_mov_b32 m0, %0"
                 : "=&s"(keep)
                 : "s"(lds), "v"(voff), "s"(rs), "s"(soff)
                 : "memory");
}

// The slot barrier: this wave's own memory operations except the N most
// recent, and all of its LDS operations, are complete; then s_barrier.  Both
// are the compiler's own builtins, so that its tracking of LDS waits sees
// them (the same instructions in an asm statement gave a different schedule
// of the slot, 6% slower on mixed widths in compact storage).
template <int N> __device__ __forceinline__ void ring_barrier()
{
    __builtin_amdgcn_s_waitcnt((N & 15) | (((N >> 4) & 3) << 14) | (7 << 4));
    __builtin_amdgcn_s_barrier();
}
// The same for a wave-uniform count n <= MAXN (the wait takes an immediate:
// one branch per possible count).
template <int MAXN> __device__ __forceinline__ void ring_barrier_n(int n)
{
    auto one = [&](auto tag) {
        constexpr int N = decltype(tag)::value;
        if constexpr (N <= MAXN) {
            if (n == N) {
                ring_barrier<N>();
                return true;
            }
        }
        return false;
    };
    if (one(std::integral_constant<int, 0>{}) || one(std::integral_constant<int, 1>{}) ||
        one(std::integral_constant<int, 2>{}) || one(std::integral_constant<int, 3>{}) ||
        one(std::integral_constant<int, 4>{}) || one(std::integral_constant<int, 5>{}) ||
        one(std::integral_constant<int, 6>{}) || one(std::integral_constant<int, 7>{}) ||
        one(std::integral_constant<int, 8>{}) || one(std::integral_constant<int, 9>{}) ||
        one(std::integral_constant<int, 10>{}) || one(std::integral_constant<int, 11>{}))
        return;
    ring_barrier<0>();
}

__device__ __forceinline__ int wcode_of(const ScanArgs &a, int k)
{
    return k >= 0 ? (int)((a.wcode[k >> 3] >> ((k & 7) * 4)) & 15u) : 0;
}

// bf16 pair parts of (x0, x1): hi = round-to-nearest, lo = the rounded
// remainder (x - hi is exact).  (The remainders by fp32 subtraction of the
// widened hi parts: no register copies, which the in-place accumulation of a
// bf16 dot product costs here, and no wait states after them.)
struct HiLo {
    uint32_t h, l;
};
__device__ __forceinline__ HiLo hilo_pair(float x0, float x1)
{
    const uint32_t h = __builtin_bit_cast(uint32_t, __builtin_convertvector(f2{x0, x1}, bf16x2));
    const f2 r = {x0 - bitsf(h << 16), x1 - bitsf(h & kHighHalf)};
    const uint32_t l = __builtin_bit_cast(uint32_t, __builtin_convertvector(r, bf16x2));
    return {h, l};
}

__device__ __forceinline__ f4 mfma_bf16(const bf16x8 &a, const bf16x8 &b, const f4 &c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Pn = A_j P_{j+1} for NR row blocks and NKP 32-wide k blocks (the live part
// of tile j) over this wave's CB column blocks, and with AFF the raw c rows
// of this wave's row blocks I = w + NW ii: Cn[ii] = A_j c_{j+1} (their A
// operands read once more).  ring: LDS byte address of the tile's first
// block plus this lane's operand offset; cop: of the bf16 parts of c_{j+1}
// for this lane's k values.  P is consumed.
template <int NW, int NR, int NKP, bool AFF>
__device__ __forceinline__ void ring_combine(f4 (&Pn)[8][4 / NW], f4 (&P)[8][4 / NW],
                                             f4 (&Cn)[8 / NW], uint32_t ring, uint32_t cop, int w)
{
    constexpr int CB = 4 / NW;
    typedef __attribute__((address_space(3))) char lchar;
    auto rd = [](uint32_t a) { return *(const bf16x8 *)(lchar *)(uintptr_t)a; };
    const f4 z = {0.0f, 0.0f, 0.0f, 0.0f};
    // rows past r_j are never read: their registers get a new, unspecified
    // value (an empty asm defines them), so that nothing from an earlier slot
    // stays live in them and no instruction is spent
#pragma unroll
    for (int I = NR; I < 8; ++I)
#pragma unroll
        for (int t = 0; t < CB; ++t)
            asm volatile("" : "=v"(Pn[I][t]));
#pragma unroll
    for (int p = 0; p < NKP; ++p) {
        // B operands: rows 32p + 8g + 0..7 of P (blocks 2p, 2p+1 of the
        // accumulator), split into bf16 parts, per column block
        bf16x8 bh[CB], bl[CB];
#pragma unroll
        for (int t = 0; t < CB; ++t) {
            u4 hh, ll;
#pragma unroll
            for (int e = 0; e < 2; ++e) {
                const HiLo s0 = hilo_pair(P[2 * p][t][2 * e], P[2 * p][t][2 * e + 1]);
                const HiLo s1 = hilo_pair(P[2 * p + 1][t][2 * e], P[2 * p + 1][t][2 * e + 1]);
                hh[e] = s0.h;
                hh[e + 2] = s1.h;
                ll[e] = s0.l;
                ll[e + 2] = s1.l;
            }
            bh[t] = __builtin_bit_cast(bf16x8, hh);
            bl[t] = __builtin_bit_cast(bf16x8, ll);
        }
        // row blocks in pairs: two operand reads, then the hi products and
        // the lo products (independent accumulators back to back)
#pragma unroll
        for (int I = 0; I < NR; I += 2) {
            const bf16x8 a0 = rd(ring + (I * NKP + p) * kBlk);
            const bf16x8 a1 = rd(ring + ((I + 1) * NKP + p) * kBlk);
#pragma unroll
            for (int t = 0; t < CB; ++t) {
                Pn[I][t] = mfma_bf16(a0, bh[t], p == 0 ? z : Pn[I][t]);
                Pn[I + 1][t] = mfma_bf16(a1, bh[t], p == 0 ? z : Pn[I + 1][t]);
            }
#pragma unroll
            for (int t = 0; t < CB; ++t) {
                Pn[I][t] = mfma_bf16(a0, bl[t], Pn[I][t]);
                Pn[I + 1][t] = mfma_bf16(a1, bl[t], Pn[I + 1][t]);
            }
        }
    }
    if constexpr (AFF) {
        // c rows of row blocks w + NW ii below NR; w is wave-uniform
        constexpr int NC = NR >= NW ? NR / NW : 1;
#pragma unroll
        for (int ii = 0; ii < 8 / NW; ++ii)
            asm volatile("" : "=v"(Cn[ii]));
        if (NR >= NW || w < NR) {
            const uint32_t cring = ring + (uint32_t)(w * NKP * kBlk);
#pragma unroll
            for (int p = 0; p < NKP; ++p) {
                const bf16x8 ch = rd(cop + 64 * p);
                const bf16x8 cl = rd(cop + 256 + 64 * p);
#pragma unroll
                for (int ii = 0; ii < NC; ++ii) {
                    const bf16x8 a = rd(cring + (NW * ii * NKP + p) * kBlk);
                    Cn[ii] = mfma_bf16(a, ch, p == 0 ? z : Cn[ii]);
                    Cn[ii] = mfma_bf16(a, cl, Cn[ii]);
                }
            }
        }
    }
}

// The combine of slot j for its runtime shape (row blocks nr of 2, 4, 8; k
// blocks nkp of 1, 2, 4); only the shapes of at most MAXB blocks are built.
template <int NW, int RMAX, int MAXB, bool AFF>
__device__ __forceinline__ void ring_combine_shape(int nr, int nkp, f4 (&Pn)[8][4 / NW],
                                                   f4 (&P)[8][4 / NW], f4 (&Cn)[8 / NW],
                                                   uint32_t ring, uint32_t cop, int w)
{
#define LBI_RING_CASE(NR, NKP)                                               \
    if constexpr (NR * NKP <= MAXB && 16 * NR <= RMAX && 32 * NKP <= RMAX) \
        if (nr == NR && nkp == NKP) {                                        \
            ring_combine<NW, NR, NKP, AFF>(Pn, P, Cn, ring, cop, w);         \
            return;                                                          \
        }
    LBI_RING_CASE(2, 1)
    LBI_RING_CASE(2, 2)
    LBI_RING_CASE(4, 1)
    LBI_RING_CASE(4, 2)
    LBI_RING_CASE(2, 4)
    LBI_RING_CASE(4, 4)
    LBI_RING_CASE(8, 1)
    LBI_RING_CASE(8, 2)
    LBI_RING_CASE(8, 4)
#undef LBI_RING_CASE
}

// (NW: waves per chain, 4 or 2, each owning 4 / NW of the composite's four
// column blocks; RMAX: largest width; MAXB: most blocks in a tile, 8 or 16;
// AFF: b present; COMPACT: tiles at their true shapes back to back, else
// zero-padded RMAX x RMAX)
// (launch bounds: four chains per CU are NW waves per SIMD)
template <int NW, int RMAX, int MAXB, bool AFF, bool COMPACT>
__global__ __launch_bounds__(64 * NW, NW) void scan_ring_kernel(const ScanArgs args)
{
    extern __shared__ __attribute__((aligned(16))) char lds_dyn[];
    typedef __attribute__((address_space(3))) char lchar;
    const uint32_t lbase = (uint32_t)(uintptr_t)(lchar *)lds_dyn;
    auto lptr = [](uint32_t addr) { return (lchar *)(uintptr_t)addr; };

    constexpr int CB = 4 / NW;                    // column blocks per wave
    constexpr int DPW = MAXB / NW;                // most block loads per wave and slot
    // (most memory operations newer than a tile's: the next tile's loads, its
    // b load and two lambda stores)
    constexpr int MAXN = DPW + 3;
    const int ring = args.ring;
    const RingLds lo = ring_lds(ring, AFF);
    const int pitch = args.pitch;                 // padded storage: RMAX

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
    const int g = lane >> 4;
    const int li = lane & 15;
    const int64_t beta = blockIdx.x;
    const int K = (int)args.K;  // at most LBI_MAX_HINT_K

    // ---- per-chain buffers (one resource each) --------------------------------
    const __bf16 *Ach = (const __bf16 *)args.A +
                        (COMPACT ? beta * (int64_t)args.totalA : beta * K * (int64_t)(pitch * pitch));
    const i4 rsA = rsrc(Ach, (uint32_t)(COMPACT ? args.totalA * 2 : K * pitch * pitch * 2));
    const __bf16 *bch = AFF ? (const __bf16 *)args.b +
                                  (COMPACT ? beta * (int64_t)args.totalR : beta * K * (int64_t)pitch)
                            : nullptr;
    const i4 rsB = rsrc(bch, AFF ? (uint32_t)(COMPACT ? args.totalR * 2 : K * pitch * 2) : 0u);
    float *lch = args.lam + (COMPACT ? beta * (int64_t)args.totalR : beta * K * (int64_t)pitch);
    const __amdgpu_buffer_rsrc_t rsL = __builtin_amdgcn_make_buffer_rsrc(
        lch, 0, (int)(COMPACT ? args.totalR * 4 : K * pitch * 4), kBufferWord3);
    int32_t curA = args.totalA, curB = args.totalR, curL = args.totalR;  // compact offsets

    // ---- per-lane constants ---------------------------------------------------
    // operand read: row li of a block, natural chunk g at slot g ^ (li / 4)
    const uint32_t opoff = (uint32_t)(li * 64 + ((g ^ (li >> 2)) & 3) * 16);
    // block load: lane -> LDS row dr = lane / 4, slot lane % 4 holding
    // natural chunk dq; tile row 32 (I / 2) + 4 (I % 2) + drow
    const int dr = lane >> 2;
    const int dq = (lane & 3) ^ ((dr >> 2) & 3);
    const int drow = 8 * (dr >> 2) + (dr & 3);
    const int vpad = (drow * pitch + 8 * dq) * 2;  // zero-padded storage
    // lambda_K at this lane's columns 16 (w + NW t) + li
    float lk[CB];
#pragma unroll
    for (int t = 0; t < CB; ++t)
        lk[t] = (float)((const __bf16 *)args.lamK)[beta * (COMPACT ? 64 : pitch) +
                                                   16 * (w + NW * t) + li];

    // ---- issue tile t (codes rc = r_t / 16, cc = r_{t+1} / 16) at ring block
    // base, and b_t; returns the number of loads this wave issued ----------
    // Load d of this wave in a slot is block NW d + w of the tile,
    // at row block I = (NW d + w) / nkp and k block p = (NW d + w) mod nkp
    // (nkp = 1, 2, 4: the tile's 32-wide k blocks); its first tile row is
    // 32 (I / 2) + 4 (I % 2).  (Shifts only: a select among precomputed
    // values per nkp becomes a table in private memory.)
    // (bsl: the b slot of tile t; slots 0, 1, 2 in the order tiles are issued)
    auto issue = [&](int t, int base, int rc, int cc, int bsl) {
        const bool live = t >= 0;
        const int nkp = cc >> 1;          // 1, 2 or 4 k blocks
        const int c = nkp >> 1;           // log2(nkp)
        const int nblk = live ? rc * nkp : 0;
        int tile_off;  // byte offset of the tile in the chain's A
        int cols;      // row pitch in elements
        if constexpr (COMPACT) {
            if (live)
                curA -= rc * 16 * cc * 16;
            tile_off = curA * 2;
            cols = cc * 16;
        } else {
            tile_off = (live ? t : 0) * pitch * pitch * 2;
            cols = pitch;
        }
        const int vbase = COMPACT ? (drow * cols + 8 * dq) * 2 : vpad;
        const uint32_t mrow = lbase + (uint32_t)((base + w) * kBlk);
        int n = 0;
#pragma unroll
        for (int d = 0; d < DPW; ++d) {
            const int bk = NW * d + w;
            if (bk < nblk) {
                const int I = bk >> c, p = bk & (nkp - 1);
                dma_b128(mrow + (uint32_t)(NW * d * kBlk), rsA, vbase,
                         tile_off + ((32 * (I >> 1) + 4 * (I & 1)) * cols + 32 * p) * 2);
                ++n;
            }
        }
        if constexpr (AFF) {
            // b_t: 64 lanes x 4 bytes (2 values each) by wave 0, into b slot
            // bsl
            const int rows = live ? rc * 16 : 0;
            int soffb;
            if constexpr (COMPACT) {
                curB -= rows;
                soffb = curB * 2;
            } else {
                soffb = (live ? t : 0) * pitch * 2;
            }
            if (w == 0 && live) {
                dma_b32(lbase + (uint32_t)(lo.b + bsl * 256), rsB,
                        2 * lane < rows ? lane * 4 : kOutOfRange, soffb);
                ++n;
            }
        }
        return n;
    };

    // ---- lambda_s = sum of the wave partials + c_s, stored by two waves -------
    // (one buffer store per wave, out of range for lanes with nothing to store;
    // with four waves the pair s % 2 stores)
    auto finalize = [&](int s, bool valid, int rc) {
        const int row = NW == 4 ? tid - 128 * (s & 1) : tid;
        const bool mine = valid && row >= 0 && row < 128;
        const int rr = mine ? row : 0;
        const int rows = valid ? rc * 16 : 0;
        float acc = 0.0f;
        const float *part = (const float *)lptr(lbase + lo.part + (s & 1) * 4 * 128 * 4);
        if (rr < rows) {
            acc = part[rr] + part[128 + rr];
            if constexpr (NW == 4)
                acc += part[256 + rr] + part[384 + rr];
            if constexpr (AFF)
                acc += ((const float *)lptr(lbase + lo.c + (s & 3) * 512))[rr];
        }
        int soff;
        if constexpr (COMPACT) {
            if (valid)
                curL -= rows;
            soff = curL * 4;
        } else {
            soff = (valid ? s : 0) * pitch * 4;
        }
        // (zero-padded storage: rows r_s .. pitch - 1 are written as 0)
        __builtin_amdgcn_raw_buffer_store_b32(
            __float_as_uint(acc), rsL,
            mine && rr < (COMPACT ? rows : (valid ? pitch : 0)) ? rr * 4 : kOutOfRange, soff, 0);
    };

    // ---- partial P lambda_K over this wave's columns, rows of nb blocks ------
    // (row blocks I0 .. I0 + NB - 1; at most four at a time)
    auto apply_nb = [&](const f4 (&P)[8][CB], int pbuf, auto nb_tag, auto i0_tag) {
        constexpr int NB = decltype(nb_tag)::value;
        constexpr int I0 = decltype(i0_tag)::value;
        constexpr int LIVE = 4 * NB;
        float q[LIVE];
#pragma unroll
        for (int I = 0; I < NB; ++I)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                float x = P[I0 + I][0][v] * lk[0];
#pragma unroll
                for (int t = 1; t < CB; ++t)
                    x += P[I0 + I][t][v] * lk[t];
                q[4 * I + v] = x;
            }
        group_reduce<16, LIVE>(q, li);
        float *part = (float *)lptr(lbase + lo.part + pbuf * 4 * 128 * 4 + w * 128 * 4);
        if constexpr (LIVE >= 16) {
            const int idx = li;  // = 4 I + v
            part[sigma_row(I0 + (idx >> 2), 4 * g + (idx & 3))] = q[0];
        } else {
            const int idx = li >> 1;
            if ((li & 1) == 0)
                part[sigma_row(I0 + (idx >> 2), 4 * g + (idx & 3))] = q[0];
        }
    };
    using C0 = std::integral_constant<int, 0>;
    using C2 = std::integral_constant<int, 2>;
    using C4 = std::integral_constant<int, 4>;
    auto apply = [&](const f4 (&P)[8][CB], int pbuf, int nb) {
        if (nb <= 2) {
            apply_nb(P, pbuf, C2{}, C0{});
        } else {
            apply_nb(P, pbuf, C4{}, C0{});
            if constexpr (RMAX == 128)
                if (nb > 4)
                    apply_nb(P, pbuf, C4{}, C4{});
        }
    };

    // ---- c_j = (raw rows of this wave's c blocks) + b_j, to LDS ---------------
    // lane (li < 4 NC): value v = li % 4 of its ii-th c block (ii = li / 4,
    // row block I = w + NW ii) at rows 4 g + v of the block, i.e. tile row
    // sigma_row(I, 4 g + v)
    // (bsl: the b slot of slot j)
    auto c_out = [&](int j, int nr, const f4 (&Cn)[8 / NW], bool from_b_only, int bsl) {
        if constexpr (AFF) {
            const int v = li & 3, ii = li >> 2;
            const int I = w + NW * ii;
            if (ii < 8 / NW && I < nr) {
                float x = 0.0f;
                if (!from_b_only) {
                    // (selects on values: no indexing of the register array)
                    auto pick = [&](const f4 &c4) {
                        const float x0 = v & 1 ? c4[1] : c4[0], x1 = v & 1 ? c4[3] : c4[2];
                        return v & 2 ? x1 : x0;
                    };
                    x = pick(Cn[0]);
#pragma unroll
                    for (int k = 1; k < 8 / NW; ++k)
                        if (ii == k)
                            x = pick(Cn[k]);
                }
                const int row = sigma_row(I, 4 * g + v);
                const __bf16 bv = ((const __bf16 *)lptr(lbase + lo.b + bsl * 256))[row];
                const float c = x + (float)bv;
                ((float *)lptr(lbase + lo.c + (j & 3) * 512))[row] = c;
                const __bf16 h = (__bf16)c;
                const __bf16 l = (__bf16)(c - (float)h);
                __bf16 *cop = (__bf16 *)lptr(lbase + lo.cop + (j & 1) * 512);
                cop[row] = h;
                cop[128 + row] = l;
            }
        }
    };

    // ---- prologue: tiles K-1 and K-2 in flight, then K-3 -----------------------
    // width codes of slots j+2 .. j-3 for the first step (j = K-2)
    // (packed: code d in bits 4d .. 4d + 3)
    uint32_t wqp = 0;
#pragma unroll
    for (int d = 0; d < 6; ++d)
        wqp |= (uint32_t)wcode_of(args, K - d) << (4 * d);
    auto wq = [&](int d) { return (int)((wqp >> (4 * d)) & 15u); };
    // ring block bases of tiles j, j-1, j-2 (allocation: right after the
    // previous tile, or from block 0 when the ring end would be passed)
    auto next_base = [&](int prev, int nprev, int n) {
        return prev + nprev + n <= ring ? prev + nprev : 0;
    };
    const int n_k1 = wq(1) * (wq(0) >> 1);  // blocks of tile K-1
    const int n_k2 = wq(2) * (wq(1) >> 1);
    const int n_k3 = wq(3) * (wq(2) >> 1);
    // (tJ, tJ1: bases of the tiles j and j-1 of the step about to run)
    int tJ = next_base(0, n_k1, n_k2);            // tile K-2 (tile K-1 at block 0)
    int tJ1 = next_base(tJ, n_k2, n_k3);          // tile K-3
    // Each slot barrier waits until this wave's loads of tile j (and b_j)
    // are done: its memory operations newer than those are the loads of tile
    // j-1 (cnt1 of them) and two lambda stores.
    issue(K - 1, 0, wq(1), wq(0), 0);
    const int cnt_k2 = issue(K - 2, tJ, wq(2), wq(1), 1);
    ring_barrier_n<MAXN>(cnt_k2);
    int cnt1 = issue(K - 3, tJ1, wq(3), wq(2), 2);
    // two stores that write nothing stand for the lambda stores of the two
    // slots before the first
    {
        const __amdgpu_buffer_rsrc_t none = __builtin_amdgcn_make_buffer_rsrc(lch, 0, 0, kBufferWord3);
        __builtin_amdgcn_raw_buffer_store_b32(0u, none, kOutOfRange, 0, 0);
        __builtin_amdgcn_raw_buffer_store_b32(0u, none, kOutOfRange, 0, 0);
    }

    f4 P[8][CB], Pn[8][CB], Cn[8 / NW];
    {
        // P_{K-1} = A_{K-1}: column col = 16 (w + NW t) + li is chunk
        // (col % 32) / 8 of k block col / 32; LDS row 4 g + v of each row block
        const int nr = wq(1), nkp = wq(0) >> 1;
#pragma unroll
        for (int t = 0; t < CB; ++t) {
            const int col = 16 * (w + NW * t) + li;
            const int q = (col & 31) >> 3;
#pragma unroll
            for (int I = 0; I < 8; ++I)
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    float x = 0.0f;
                    if (I < nr && (RMAX == 128 || I < 4)) {
                        const int r = 4 * g + v;
                        const uint32_t a =
                            lbase + (uint32_t)((I * nkp + (col >> 5)) * kBlk + r * 64 +
                                               ((q ^ (r >> 2)) & 3) * 16 + (col & 7) * 2);
                        x = (float)*(const __bf16 *)lptr(a);
                    }
                    P[I][t][v] = x;
                }
        }
#pragma unroll
        for (int ii = 0; ii < 8 / NW; ++ii)
            Cn[ii] = f4{0.0f, 0.0f, 0.0f, 0.0f};
        c_out(K - 1, wq(1), Cn, true, 0);
    }

    // ---- slots K-2 .. 0 ---------------------------------------------------------
    // Step j: barrier (tile j and b_j landed; the buffers written last step
    // visible); load tile j-2 into the blocks tile j+1 held; store lambda_{j+2};
    // partial apply of P_{j+1}; P_j, c_j from tile j; c_j to LDS.
    int bs = 1;  // b slot of tile j (tile K-1 took slot 0)
    // the code that enters the window at the end of step j (slot j - 4),
    // read a step early: its scalar load is complete by the next barrier
    uint32_t wpend = (uint32_t)wcode_of(args, K - 6);
    auto step = [&](int j, f4 (&Pc)[8][CB], f4 (&Pnext)[8][CB]) {
        const uint32_t wnext = (uint32_t)wcode_of(args, j - 5);
        ring_barrier_n<MAXN>(cnt1 + 2);
        const int n_j1 = wq(3) * (wq(2) >> 1), n_j2 = wq(4) * (wq(3) >> 1);
        const int bNew = next_base(tJ1, n_j1, n_j2);   // tile j-2
        // (b slots: tile j's is bs, the tile issued now takes the one
        // tile j+1 held)
        cnt1 = issue(j - 2, bNew, wq(4), wq(3), bs == 0 ? 2 : bs - 1);
        finalize(j + 2, j + 2 <= K - 1, wq(0));
        apply(Pc, (j + 1) & 1, wq(1));
        // (the apply's reads of P_{j+1} stay ahead of the combine, which
        // consumes P_{j+1}'s registers)
        __builtin_amdgcn_sched_barrier(0);
        const uint32_t cop = lbase + (uint32_t)(lo.cop + ((j + 1) & 1) * 512 + 16 * g);
        ring_combine_shape<NW, RMAX, MAXB, AFF>(wq(2), wq(1) >> 1, Pnext, Pc, Cn,
                                                lbase + (uint32_t)(tJ * kBlk) + opoff, cop, w);
        c_out(j, wq(2), Cn, false, bs);
        bs = bs == 2 ? 0 : bs + 1;
        // roll the windows by one slot
        tJ = tJ1;
        tJ1 = bNew;
        wqp = (wqp >> 4) | (wpend << 20);
        wpend = wnext;
    };
    int j = K - 2;
    for (; j >= 1; j -= 2) {
        step(j, P, Pn);
        step(j - 1, Pn, P);
    }
    if (j == 0) {
        step(0, P, Pn);
#pragma unroll
        for (int I = 0; I < 8; ++I)
#pragma unroll
            for (int t = 0; t < CB; ++t)
                P[I][t] = Pn[I][t];
    }

    // ---- the last two slots -----------------------------------------------------
    // (after the loop wq(0) is the code of slot 1, wq(1) of slot 0)
    ring_barrier<63>();
    if (K >= 2)
        finalize(1, true, wq(0));
    apply(P, 0, wq(1));
    ring_barrier<63>();
    finalize(0, true, wq(1));
}

}  // namespace

// ---- host side ----------------------------------------------------------------

namespace {
template <int NW, int RMAX, int MAXB, bool AFF, bool COMPACT>
hipError_t launch_ring_kernel(const ChainLaunch &c)
{
    void *params[] = {(void *)&c.args};
    const RingLds lo = ring_lds(c.args.ring, AFF);
    return hipLaunchKernel((const void *)&scan_ring_kernel<NW, RMAX, MAXB, AFF, COMPACT>,
                           dim3((unsigned)c.B), dim3(64 * NW), params, (size_t)lo.total,
                           c.stream);
}
template <int NW, int RMAX, int MAXB> hipError_t launch_ring_r(const ChainLaunch &c)
{
    if (c.args.compact)
        return c.aff ? launch_ring_kernel<NW, RMAX, MAXB, true, true>(c)
                     : launch_ring_kernel<NW, RMAX, MAXB, false, true>(c);
    return c.aff ? launch_ring_kernel<NW, RMAX, MAXB, true, false>(c)
                 : launch_ring_kernel<NW, RMAX, MAXB, false, false>(c);
}
}  // namespace

int ring_lds_bytes(int ring, bool aff) { return ring_lds(ring, aff).total; }

hipError_t launch_chain_ring_bf16(const ChainLaunch &c, int maxb)
{
    // (waves per chain: two at width 128, four at 64)
    if (c.r == 64 && maxb == 8)
        return launch_ring_r<LBI_RING_NW64, 64, 8>(c);
    if (c.r == 128 && maxb == 16)
        return launch_ring_r<LBI_RING_NW128, 128, 16>(c);
    return hipErrorInvalidValue;
}

}  // namespace lbi
