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
//     memory count (every wave issues the same number of memory operations
//     per slot: DPW block loads, one b load, one lambda store).
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
//     back as bf16 hi + lo (or rounded once); wave w owns column block w.
//   * c_j = A_j c_{j+1} + b_j on the matrix cores as well: c_{j+1} (hi + lo,
//     the same value in all 16 columns of a B operand) against the A operands
//     already read for P, row block I by wave I % 4.  The wave then adds b_j
//     to its rows and writes c_j (fp32, for lambda) and its bf16 parts (the
//     next slot's operand) to LDS.
//   * lambda_j: per-wave partial P_{j+1} lambda_K (a DPP butterfly over the
//     16 lanes of a column block), summed across the waves through LDS with
//     c_j and stored once, coalesced, by a pair of waves.
//
// All HIP code here is built with packed fp32 math disabled.

#include "lbi_device.hpp"
#include "lbi_internal.h"

namespace lbi {
namespace {

typedef int i4 __attribute__((ext_vector_type(4)));

constexpr int kBlk = 1024;  // bytes of one 16-row x 32-column bf16 block

// Dynamic LDS layout (bytes) for a ring of `ring` blocks.
struct RingLds {
    int dummy, part, c, cop, b, total;
};
__host__ __device__ constexpr RingLds ring_lds(int ring, bool aff)
{
    RingLds o{};
    o.dummy = ring * kBlk;            // target of loads for absent blocks
    o.part = o.dummy + kBlk;          // [2][4 waves][128] fp32 partial applies
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

// The loads of one slot: DPW block loads (16 bytes per lane, lane l's bytes
// to LDS m0[d] + 16 l) and, with B32, one 4-byte load per lane (to
// m0b + 4 l).  M0 holds each LDS destination in turn (one wait state after
// writing it); its value from before is restored at the end.
template <int DPW, bool B32>
__device__ __forceinline__ void dma_slot(const uint32_t (&m0)[DPW], const int (&voff)[DPW],
                                         const int (&soff)[DPW], i4 rs, uint32_t m0b, int voffb,
                                         int soffb, i4 rsb)
{
    uint32_t keep;
    if constexpr (DPW == 2 && !B32) {
        asm volatile(
            "s_mov_b32 %0, m0\n\t"
            "s_mov_b32 m0, %1\n\ts_nop 0\n\tbuffer_load_dwordx4 %3, %5, %6 offen lds\n\t"
            "s_mov_b32 m0, %2\n\ts_nop 0\n\tbuffer_load_dwordx4 %4, %5, %7 offen lds\n\t"
            "s_mov_b32 m0, %0"
            : "=&s"(keep)
            : "s"(m0[0]), "s"(m0[1]), "v"(voff[0]), "v"(voff[1]), "s"(rs), "s"(soff[0]),
              "s"(soff[1])
            : "memory");
    } else if constexpr (DPW == 2 && B32) {
        asm volatile(
            "s_mov_b32 %0, m0\n\t"
            "s_mov_b32 m0, %1\n\ts_nop 0\n\tbuffer_load_dwordx4 %4, %6, %7 offen lds\n\t"
            "s_mov_b32 m0, %2\n\ts_nop 0\n\tbuffer_load_dwordx4 %5, %6, %8 offen lds\n\t"
            "s_mov_b32 m0, %3\n\ts_nop 0\n\tbuffer_load_dword %9, %10, %11 offen lds\n\t"
            "s_mov_b32 m0, %0"
            : "=&s"(keep)
            : "s"(m0[0]), "s"(m0[1]), "s"(m0b), "v"(voff[0]), "v"(voff[1]), "s"(rs),
              "s"(soff[0]), "s"(soff[1]), "v"(voffb), "s"(rsb), "s"(soffb)
            : "memory");
    } else if constexpr (DPW == 4 && !B32) {
        asm volatile(
            "s_mov_b32 %0, m0\n\t"
            "s_mov_b32 m0, %1\n\ts_nop 0\n\tbuffer_load_dwordx4 %5, %9, %10 offen lds\n\t"
            "s_mov_b32 m0, %2\n\ts_nop 0\n\tbuffer_load_dwordx4 %6, %9, %11 offen lds\n\t"
            "s_mov_b32 m0, %3\n\ts_nop 0\n\tbuffer_load_dwordx4 %7, %9, %12 offen lds\n\t"
            "s_mov_b32 m0, %4\n\ts_nop 0\n\tbuffer_load_dwordx4 %8, %9, %13 offen lds\n\t"
            "s_mov_b32 m0, %0"
            : "=&s"(keep)
            : "s"(m0[0]), "s"(m0[1]), "s"(m0[2]), "s"(m0[3]), "v"(voff[0]), "v"(voff[1]),
              "v"(voff[2]), "v"(voff[3]), "s"(rs), "s"(soff[0]), "s"(soff[1]), "s"(soff[2]),
              "s"(soff[3])
            : "memory");
    } else {
        static_assert(DPW == 4 && B32, "block loads per slot");
        asm volatile(
            "s_mov_b32 %0, m0\n\t"
            "s_mov_b32 m0, %1\n\ts_nop 0\n\tbuffer_load_dwordx4 %6, %10, %11 offen lds\n\t"
            "s_mov_b32 m0, %2\n\ts_nop 0\n\tbuffer_load_dwordx4 %7, %10, %12 offen lds\n\t"
            "s_mov_b32 m0, %3\n\ts_nop 0\n\tbuffer_load_dwordx4 %8, %10, %13 offen lds\n\t"
            "s_mov_b32 m0, %4\n\ts_nop 0\n\tbuffer_load_dwordx4 %9, %10, %14 offen lds\n\t"
            "s_mov_b32 m0, %5\n\ts_nop 0\n\tbuffer_load_dword %15, %16, %17 offen lds\n\t"
            "s_mov_b32 m0, %0"
            : "=&s"(keep)
            : "s"(m0[0]), "s"(m0[1]), "s"(m0[2]), "s"(m0[3]), "s"(m0b), "v"(voff[0]),
              "v"(voff[1]), "v"(voff[2]), "v"(voff[3]), "s"(rs), "s"(soff[0]), "s"(soff[1]),
              "s"(soff[2]), "s"(soff[3]), "v"(voffb), "s"(rsb), "s"(soffb)
            : "memory");
    }
}
// The slot barrier: this wave's own memory operations except the N most
// recent, and all of its LDS operations, are complete; then s_barrier.  The
// asm is also a compiler barrier for memory accesses.
template <int N> __device__ __forceinline__ void ring_barrier()
{
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" : : "n"(N) : "memory");
}

__device__ __forceinline__ int wcode_of(const ScanArgs &a, int k)
{
    return k >= 0 ? (int)((a.wcode[k >> 3] >> ((k & 7) * 4)) & 15u) : 0;
}

// bf16 pair parts of (x0, x1): hi = round-to-nearest, lo = the rounded
// remainder (x - hi is exact: one bf16 dot product with (-1, 0) / (0, -1));
// x0 and x1 are consumed.
// (sel: the bf16 pairs (-1, 0) and (0, -1), held in registers: an inline
// constant in a packed bf16 operand is not read as a bf16 pair)
struct HiLo {
    uint32_t h, l;
};
struct Sel {
    bf16x2 s0, s1;
};
// (The dot product accumulates into x's register: x must be dead after it,
// or the compiler copies it first.)
__device__ __forceinline__ HiLo hilo_pair(float x0, float x1, const Sel &sel)
{
    const bf16x2 h = __builtin_convertvector(f2{x0, x1}, bf16x2);
    const float r0 = __builtin_amdgcn_fdot2_f32_bf16(h, sel.s0, x0, false);
    const float r1 = __builtin_amdgcn_fdot2_f32_bf16(h, sel.s1, x1, false);
    const bf16x2 l = __builtin_convertvector(f2{r0, r1}, bf16x2);
    return {__builtin_bit_cast(uint32_t, h), __builtin_bit_cast(uint32_t, l)};
}

__device__ __forceinline__ f4 mfma_bf16(const bf16x8 &a, const bf16x8 &b, const f4 &c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Pn = A_j P_{j+1} for NR row blocks and NKP 32-wide k blocks (the live part
// of tile j), and with AFF the raw c rows of this wave's row blocks
// I = w + 4 ii: Cn[ii] = A_j c_{j+1} (their A operands read once more).
// ring: LDS byte address of the tile's first block plus this lane's operand
// offset; cop: of the bf16 parts of c_{j+1} for this lane's k values.  P is
// consumed.
template <int NR, int NKP, bool AFF, bool R1>
__device__ __forceinline__ void ring_combine(f4 (&Pn)[8], f4 (&P)[8], f4 (&Cn)[2], uint32_t ring,
                                             uint32_t cop, int w, const Sel &sel)
{
    typedef __attribute__((address_space(3))) char lchar;
    auto rd = [](uint32_t a) { return *(const bf16x8 *)(lchar *)(uintptr_t)a; };
    const f4 z = {0.0f, 0.0f, 0.0f, 0.0f};
    // rows past r_j are never read: their registers get a new, unspecified
    // value (an empty asm defines them), so that nothing from an earlier slot
    // stays live in them and no instruction is spent
#pragma unroll
    for (int I = NR; I < 8; ++I)
        asm volatile("" : "=v"(Pn[I]));
#pragma unroll
    for (int p = 0; p < NKP; ++p) {
        // B operand: rows 32p + 8g + 0..7 of P (blocks 2p, 2p+1 of the
        // accumulator), split into bf16 parts
        u4 hh, ll;
#pragma unroll
        for (int e = 0; e < 2; ++e) {
            const HiLo s0 = hilo_pair(P[2 * p][2 * e], P[2 * p][2 * e + 1], sel);
            const HiLo s1 = hilo_pair(P[2 * p + 1][2 * e], P[2 * p + 1][2 * e + 1], sel);
            hh[e] = s0.h;
            hh[e + 2] = s1.h;
            ll[e] = s0.l;
            ll[e + 2] = s1.l;
        }
        const bf16x8 bh = __builtin_bit_cast(bf16x8, hh);
        const bf16x8 bl = __builtin_bit_cast(bf16x8, ll);
        // row blocks in pairs: two operand reads, then the two hi products
        // and the two lo products (independent accumulators back to back)
#pragma unroll
        for (int I = 0; I < NR; I += 2) {
            const bf16x8 a0 = rd(ring + (I * NKP + p) * kBlk);
            const bf16x8 a1 = rd(ring + ((I + 1) * NKP + p) * kBlk);
            Pn[I] = mfma_bf16(a0, bh, p == 0 ? z : Pn[I]);
            Pn[I + 1] = mfma_bf16(a1, bh, p == 0 ? z : Pn[I + 1]);
            if constexpr (!R1) {
                Pn[I] = mfma_bf16(a0, bl, Pn[I]);
                Pn[I + 1] = mfma_bf16(a1, bl, Pn[I + 1]);
            }
        }
    }
    if constexpr (AFF) {
        // c rows of row blocks w, w + 4 (those below NR); w is wave-uniform
        constexpr int NC = NR > 4 ? 2 : 1;
        asm volatile("" : "=v"(Cn[0]));
        asm volatile("" : "=v"(Cn[1]));
        if (NR >= 4 || w < NR) {
            const uint32_t cring = ring + (uint32_t)(w * NKP * kBlk);
#pragma unroll
            for (int p = 0; p < NKP; ++p) {
                const bf16x8 ch = rd(cop + 64 * p);
                const bf16x8 cl = rd(cop + 256 + 64 * p);
#pragma unroll
                for (int ii = 0; ii < NC; ++ii) {
                    const bf16x8 a = rd(cring + (4 * ii * NKP + p) * kBlk);
                    Cn[ii] = mfma_bf16(a, ch, p == 0 ? z : Cn[ii]);
                    Cn[ii] = mfma_bf16(a, cl, Cn[ii]);
                }
            }
        }
    }
}

// The combine of slot j for its runtime shape (row blocks nr of 2, 4, 8; k
// blocks nkp of 1, 2, 4).
// (only the shapes of at most 4 DPW blocks are built)
template <int RMAX, int DPW, bool AFF, bool R1>
__device__ __forceinline__ void ring_combine_shape(int nr, int nkp, f4 (&Pn)[8], f4 (&P)[8],
                                                   f4 (&Cn)[2], uint32_t ring, uint32_t cop, int w,
                                                   const Sel &sel)
{
#define LBI_RING_CASE(NR, NKP)                                            \
    if constexpr (NR * NKP <= 4 * DPW && 16 * NR <= RMAX && 32 * NKP <= RMAX) \
        if (nr == NR && nkp == NKP) {                                     \
            ring_combine<NR, NKP, AFF, R1>(Pn, P, Cn, ring, cop, w, sel); \
            return;                                                       \
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

// (RMAX: largest width; AFF: b present; COMPACT: tiles at their true shapes
// back to back, else zero-padded RMAX x RMAX; DPW: block loads per wave and
// slot, a quarter of the largest tile's blocks)
template <int RMAX, bool AFF, bool COMPACT, int DPW>
__global__ __launch_bounds__(256, 4) void scan_ring_kernel(const ScanArgs args)
{
    extern __shared__ __attribute__((aligned(16))) char lds_dyn[];
    typedef __attribute__((address_space(3))) char lchar;
    const uint32_t lbase = (uint32_t)(uintptr_t)(lchar *)lds_dyn;
    auto lptr = [](uint32_t addr) { return (lchar *)(uintptr_t)addr; };

    constexpr bool R1 = false;
    constexpr int NBO = AFF ? 1 : 0;              // b loads per wave and slot
    constexpr int NSTEP = DPW + NBO + 1;          // memory operations per wave and slot
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
    Sel sel;
    {
        uint32_t s0 = 0x0000BF80u, s1 = 0xBF800000u;
        asm("" : "+v"(s0), "+v"(s1));
        sel.s0 = __builtin_bit_cast(bf16x2, s0);
        sel.s1 = __builtin_bit_cast(bf16x2, s1);
    }
    const float lk = [&] {
        const int rK = COMPACT ? 64 : pitch;
        return (float)((const __bf16 *)args.lamK)[beta * rK + 16 * w + li];
    }();

    // b_t sits in b slot (K - 1 - t) mod 3 (t = K-1, K-2, ... in turn)
    auto bslot = [&](int t) { return (int)((uint32_t)(K - 1 - t) % 3u); };

    // ---- issue tile t (codes rc = r_t / 16, cc = r_{t+1} / 16) at ring block
    // base, and b_t: DPW + NBO memory operations per wave, whatever t --------
    // Block d of this wave's loads in a slot is block 4 d + w of the tile,
    // at row block I = (4 d + w) / nkp and k block p = w mod nkp (nkp = 1,
    // 2, 4: the tile's 32-wide k blocks); its first tile row
    // 32 (I / 2) + 4 (I % 2) is, for nkp = 4, 2, 1:
    //   32 (d / 2) + 4 (d % 2),  32 d + 4 (w / 2),  64 d + 32 (w / 2) + 4 (w % 2).
    const int wrow2 = 4 * (w >> 1), wrow1 = 32 * (w >> 1) + 4 * (w & 1);
    auto issue = [&](int t, int base, int rc, int cc) {
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
        const int poff = tile_off + 64 * (w & (nkp - 1));
        const uint32_t mrow = lbase + (uint32_t)((base + w) * kBlk);
        const uint32_t mdum = lbase + (uint32_t)lo.dummy;
        uint32_t m0[DPW];
        int voff[DPW], soff[DPW];
#pragma unroll
        for (int d = 0; d < DPW; ++d) {
            const bool real = 4 * d + w < nblk;
            // absent blocks: every lane out of range, zeros into the dummy block
            m0[d] = real ? mrow + (uint32_t)(4 * d * kBlk) : mdum;
            voff[d] = real ? vbase : kOutOfRange;
            const int r0 = c == 2 ? 32 * (d >> 1) + 4 * (d & 1)
                                  : (c == 1 ? 32 * d + wrow2 : 64 * d + wrow1);
            soff[d] = poff + r0 * cols * 2;
        }
        uint32_t m0b = mdum;
        int voffb = kOutOfRange, soffb = 0;
        if constexpr (AFF) {
            // b_t: 64 lanes x 4 bytes (2 values each) by wave 0, into b slot
            // (K - 1 - t) mod 3
            const int rows = live ? rc * 16 : 0;
            if constexpr (COMPACT) {
                curB -= rows;
                soffb = curB * 2;
            } else {
                soffb = (live ? t : 0) * pitch * 2;
            }
            const bool mine = w == 0 && live;
            if (mine)
                m0b = lbase + (uint32_t)(lo.b + bslot(t) * 256);
            voffb = mine && 2 * lane < rows ? lane * 4 : kOutOfRange;
        }
        dma_slot<DPW, AFF>(m0, voff, soff, rsA, m0b, voffb, soffb, rsB);
    };

    // ---- lambda_s = sum of the wave partials + c_s, stored by wave pair s % 2 --
    // (one buffer store per wave, out of range for lanes with nothing to store)
    auto finalize = [&](int s, bool valid, int rc) {
        const int fw = (int)(s & 1);
        const int row = tid - 128 * fw;
        const bool mine = valid && row >= 0 && row < 128;
        const int rr = mine ? row : 0;
        const int rows = valid ? rc * 16 : 0;
        float acc = 0.0f;
        const float *part = (const float *)lptr(lbase + lo.part + (int)(s & 1) * 4 * 128 * 4);
        if (rr < rows) {
            acc = (part[rr] + part[128 + rr]) + (part[256 + rr] + part[384 + rr]);
            if constexpr (AFF)
                acc += ((const float *)lptr(lbase + lo.c + (int)(s & 3) * 512))[rr];
        }
        int soff;
        if constexpr (COMPACT) {
            if (valid)
                curL -= rows;
            soff = curL * 4;
        } else {
            soff = (int)(valid ? s : 0) * pitch * 4;
        }
        // (zero-padded storage: rows r_s .. pitch - 1 are written as 0)
        __builtin_amdgcn_raw_buffer_store_b32(
            __float_as_uint(acc), rsL,
            mine && rr < (COMPACT ? rows : (valid ? pitch : 0)) ? rr * 4 : kOutOfRange, soff, 0);
    };

    // ---- partial P lambda_K over this wave's column block, rows of nb blocks --
    // (row blocks I0 .. I0 + NB - 1; at most four at a time)
    auto apply_nb = [&](const f4 (&P)[8], int pbuf, auto nb_tag, auto i0_tag) {
        constexpr int NB = decltype(nb_tag)::value;
        constexpr int I0 = decltype(i0_tag)::value;
        constexpr int LIVE = 4 * NB;
        float q[LIVE];
#pragma unroll
        for (int I = 0; I < NB; ++I)
#pragma unroll
            for (int v = 0; v < 4; ++v)
                q[4 * I + v] = P[I0 + I][v] * lk;
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
    auto apply = [&](const f4 (&P)[8], int pbuf, int nb) {
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
    // lane (li < 8): value v = li % 4 of row block I = w + 4 (li / 4) at rows
    // 4 g + v of the block, i.e. tile row sigma_row(I, 4 g + v)
    auto c_out = [&](int j, int nr, const f4 (&Cn)[2], bool from_b_only) {
        if constexpr (AFF) {
            const int v = li & 3, ii = (li >> 2) & 1;
            const int I = w + 4 * ii;
            if (li < 8 && I < nr) {
                float x = 0.0f;
                if (!from_b_only) {
                    // (selects on values: no indexing of the register array)
                    const float x0 = v & 1 ? Cn[0][1] : Cn[0][0], x1 = v & 1 ? Cn[0][3] : Cn[0][2];
                    x = v & 2 ? x1 : x0;
                    if (RMAX == 128 && ii) {
                        const float y0 = v & 1 ? Cn[1][1] : Cn[1][0], y1 = v & 1 ? Cn[1][3] : Cn[1][2];
                        x = v & 2 ? y1 : y0;
                    }
                }
                const int row = sigma_row(I, 4 * g + v);
                const __bf16 bv = ((const __bf16 *)lptr(lbase + lo.b + bslot(j) * 256))[row];
                const float c = x + (float)bv;
                ((float *)lptr(lbase + lo.c + (int)(j & 3) * 512))[row] = c;
                const __bf16 h = (__bf16)c;
                const __bf16 l = (__bf16)(c - (float)h);
                __bf16 *cop = (__bf16 *)lptr(lbase + lo.cop + (int)(j & 1) * 512);
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
    issue(K - 1, 0, wq(1), wq(0));
    issue(K - 2, tJ, wq(2), wq(1));
    ring_barrier<DPW + NBO>();
    issue(K - 3, tJ1, wq(3), wq(2));
    // one store that writes nothing, so that every slot barrier below sees
    // the same count of newer memory operations
    __builtin_amdgcn_raw_buffer_store_b32(
        0u, __builtin_amdgcn_make_buffer_rsrc(lch, 0, 0, kBufferWord3), kOutOfRange, 0, 0);

    f4 P[8], Pn[8], Cn[2];
    {
        // P_{K-1} = A_{K-1}: column 16 w + li is chunk 2 (w % 2) + li / 8 of
        // k block w / 2; LDS row 4 g + v of each row block
        const int nr = wq(1), nkp = wq(0) >> 1;
        const int q = 2 * (w & 1) + (li >> 3);
#pragma unroll
        for (int I = 0; I < 8; ++I)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                float x = 0.0f;
                if (I < nr && (RMAX == 128 || I < 4)) {
                    const int r = 4 * g + v;
                    const uint32_t a = lbase + (uint32_t)((I * nkp + (w >> 1)) * kBlk + r * 64 +
                                                          ((q ^ (r >> 2)) & 3) * 16 + (li & 7) * 2);
                    x = (float)*(const __bf16 *)lptr(a);
                }
                P[I][v] = x;
            }
        Cn[0] = Cn[1] = f4{0.0f, 0.0f, 0.0f, 0.0f};
        c_out(K - 1, wq(1), Cn, true);
    }

    // ---- slots K-2 .. 0 ---------------------------------------------------------
    // Step j: barrier (tile j and b_j landed; the buffers written last step
    // visible); load tile j-2 into the blocks tile j+1 held; store lambda_{j+2};
    // partial apply of P_{j+1}; P_j, c_j from tile j; c_j to LDS.
    auto step = [&](int j, f4 (&Pc)[8], f4 (&Pnext)[8]) {
        ring_barrier<NSTEP>();
        const int n_j1 = wq(3) * (wq(2) >> 1), n_j2 = wq(4) * (wq(3) >> 1);
        const int bNew = next_base(tJ1, n_j1, n_j2);   // tile j-2
        issue(j - 2, bNew, wq(4), wq(3));
        finalize(j + 2, j + 2 <= K - 1, wq(0));
        apply(Pc, (int)((j + 1) & 1), wq(1));
        // (the apply's reads of P_{j+1} stay ahead of the combine, which
        // consumes P_{j+1}'s registers)
        __builtin_amdgcn_sched_barrier(0);
        const uint32_t cop = lbase + (uint32_t)(lo.cop + (int)((j + 1) & 1) * 512 + 16 * g);
        ring_combine_shape<RMAX, DPW, AFF, R1>(wq(2), wq(1) >> 1, Pnext, Pc, Cn,
                                               lbase + (uint32_t)(tJ * kBlk) + opoff, cop, w, sel);
        c_out(j, wq(2), Cn, false);
        // roll the windows by one slot
        tJ = tJ1;
        tJ1 = bNew;
        wqp = (wqp >> 4) | ((uint32_t)wcode_of(args, j - 4) << 20);
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
            P[I] = Pn[I];
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
template <int RMAX, bool AFF, bool COMPACT, int DPW>
hipError_t launch_ring_kernel(const ChainLaunch &c)
{
    void *params[] = {(void *)&c.args};
    const RingLds lo = ring_lds(c.args.ring, AFF);
    return hipLaunchKernel((const void *)&scan_ring_kernel<RMAX, AFF, COMPACT, DPW>,
                           dim3((unsigned)c.B), dim3(256), params, (size_t)lo.total, c.stream);
}
template <int RMAX, int DPW> hipError_t launch_ring_r(const ChainLaunch &c)
{
    if (c.args.compact)
        return c.aff ? launch_ring_kernel<RMAX, true, true, DPW>(c)
                     : launch_ring_kernel<RMAX, false, true, DPW>(c);
    return c.aff ? launch_ring_kernel<RMAX, true, false, DPW>(c)
                 : launch_ring_kernel<RMAX, false, false, DPW>(c);
}
}  // namespace

int ring_lds_bytes(int ring, bool aff) { return ring_lds(ring, aff).total; }

hipError_t launch_chain_ring_bf16(const ChainLaunch &c, int dpw)
{
    if (c.r == 64 && dpw == 2)
        return launch_ring_r<64, 2>(c);
    if (c.r == 128 && dpw == 4)
        return launch_ring_r<128, 4>(c);
    return hipErrorInvalidValue;
}

}  // namespace lbi
