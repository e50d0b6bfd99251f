// Phase 1 of Algorithm "Bounded-Interface Backpropagation" (gfx950): the
// interface Jacobians J_k = dR_k(m_k) I_r (Eq. "jacobian-identity-
// construction") of the synthetic region map of Eq. "concrete-region-arch",
//
//   m_{k+1} = R_k(m_k) = LN(m_k + alpha_k Enc_k(pool(Phi_k(x_embed + Dec_k(m_k))))),
//   Dec_k(m) = W_d2 silu(W_d1 m + b_d1) + b_d2          (r -> D -> D)
//   Phi_k(x) = x + W2 silu(W1 x), token by token          (D -> X -> D)
//   pool     = mean over the L tokens of a sequence
//   Enc_k(p) = W_e2 silu(W_e1 p + b_e1) + b_e2          (D -> D -> r)
//   LN       = LayerNorm over the r features, gain gamma, shift beta, eps 1e-5,
//
// for every sequence b and region k at once, written as A[b][k] = J_k^T, the
// operand of the scan.
//
// The tangent of all r directions, taken exactly: Dec_k's differential
// Jdec = W_d2 diag(silu'(a)) W_d1 (D x r) is the same for every token, so
// through Phi_k and the mean pool
//   dp = Jdec + W2 diag(gbar) W1 Jdec,   gbar = mean_l silu'(W1 x_l),
// and p = mean_l x_embed + d + W2 sbar with sbar = mean_l silu(W1 x_l).  The
// per-token work is therefore one product H = X_in W1^T per sequence and region
// (L x D x X), whose epilogue reduces silu(H) and silu'(H) over the tokens; H
// never reaches memory.  The r directions then go through skinny products with
// N = B r (all sequences of a region at once) and the LayerNorm Jacobian
//   J = diag(gamma) / sigma (I - 11^T / r - zhat zhat^T / r) (I + alpha Jenc).
//
// Arithmetic: bf16 operands on the bf16 matrix cores (v_mfma_f32_16x16x32_bf16)
// with fp32 accumulation; x_embed + d and the tangent intermediates are rounded
// to bf16 (round to nearest even) where they feed a product; every vector,
// reduction and the LayerNorm part are fp32.
//
// The per-token product uses H = x_embed W1^T + 1 (W1 d)^T: x_embed is the
// same bf16 operand for every region, and d enters in fp32 through the column
// vector W1 d, added in the epilogue.
//
// Kernels, in launch order:
//   bmv x2      per region, all sequences: a -> silu(a), silu'(a); d = Dec_k(m)
//   p1          per (b, k): P1 = (diag(silu'(a)) W_d1)^T
//   bmv         cvec = W1 d
//   xpart/xfin  per b: mean_l x_embed (two-stage)
//   region_dma  per (k, b, 128 columns of X): the token product and its reductions
//   bmv x3      p = mean x_embed + d + W2 sbar; e -> silu(e), silu'(e); Enc_k
//   ln_fwd      per (b, k): z = m + alpha Enc, LayerNorm -> m_{k+1}, zhat, 1/sigma
//   gemm_nt x5  per k: Jdec^T, U'^T = (W1 Jdec)^T scaled by gbar, dp^T, T'^T, Jenc^T
//   ln_jac      per (b, k): J, stored transposed as A[b][k]

#include "lbi_device.hpp"
#include "lbi_internal.h"
#include "lbi_region_args.hpp"

namespace lbi {
namespace {

constexpr int kT = 256;
constexpr int BM = 128, BN = 128, BK = 64;
constexpr int TILE = 128 * BK;  // bf16 elements of one LDS tile (no padding)
constexpr float kLnEps = 1e-5f;

// The logistic function through the hardware reciprocal (1 ulp): it needs no
// correctly rounded division, and rcp(inf) = 0 keeps the saturated end exact.
__device__ __forceinline__ float sigm(float h) { return __builtin_amdgcn_rcpf(1.0f + __expf(-h)); }
__device__ __forceinline__ float silu(float h) { return h * sigm(h); }
__device__ __forceinline__ float dsilu(float h)
{
    const float s = sigm(h);
    return s * (1.0f + h * (1.0f - s));
}

__device__ __forceinline__ float bf(const __bf16 *p, int64_t i) { return (float)p[i]; }

__device__ __forceinline__ float wave_sum(float x)
{
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1)
        x += __shfl_xor(x, o);
    return x;
}

// ---- the tile pipeline shared by both products ---------------------------------
// LDS tile layout: 128 rows of 64 bf16 (eight 16-byte chunks), two rows per
// 256-byte line, chunk q of row R at line R / 2, slot ((R & 1) 8 + q) ^ (R / 2 & 7).
// The 16 lanes that a b128 access serves together then touch 16 distinct
// slots (all 64 banks) both when they read one chunk of 16 consecutive rows
// (an MFMA operand) and when they write the 8 chunks of 2 consecutive rows.
__device__ __forceinline__ int lds_off(int row, int q)
{
    return (row >> 1) * 128 + ((((row & 1) << 3) + q) ^ ((row >> 1) & 7)) * 8;
}

// 128 rows x 64 k of a row-major bf16 matrix (row stride ld) from row0, k0;
// rows >= nrows read as zero.  Thread t loads chunks c = t + 256 i: row c / 8,
// chunk c % 8, at the per-lane byte offsets voff (tile_offsets).  One buffer
// resource per call starts at (row0, k0) and ends with the last valid row, so
// the lanes of missing rows fall outside it and read zero (no lane masks).
__device__ __forceinline__ void tile_offsets(uint32_t (&voff)[4], int ld)
{
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int c = threadIdx.x + kT * i;
        voff[i] = (uint32_t)(((c >> 3) * ld + (c & 7) * 8) * 2);
    }
}

__device__ __forceinline__ void tile_load(u4 (&v)[4], const uint32_t (&voff)[4],
                                          const __bf16 *base, int64_t ld, int64_t row0,
                                          int64_t nrows, int k0)
{
    const int64_t left = nrows - row0;
    const int valid = left < 128 ? (int)left : 128;
    // the last valid row's chunks end at most 2 (ld - k0 - 64) bytes before
    // valid * ld * 2 - k0 * 2; the first missing row starts at or past it
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(base + row0 * ld + k0), 0, (int)(valid * (int)ld * 2 - k0 * 2), kBufferWord3);
#pragma unroll
    for (int i = 0; i < 4; ++i)
        v[i] = __builtin_amdgcn_raw_buffer_load_b128(rs, voff[i], 0, 0);
}

__device__ __forceinline__ void tile_store(const u4 (&v)[4], __bf16 *s)
{
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int c = threadIdx.x + kT * i;
        *(u4 *)(s + lds_off(c >> 3, c & 7)) = v[i];
    }
}

// ---- operands loaded straight into LDS ---------------------------------------------
typedef int i4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ i4 dma_rsrc(const void *base, uint32_t bytes)
{
    // (the values are wave-uniform; the scalar registers an asm operand of
    // class "s" needs are made explicit)
    const uint64_t x = (uint64_t)(uintptr_t)base;
    i4 v;
    v[0] = __builtin_amdgcn_readfirstlane((int)(uint32_t)x);
    v[1] = __builtin_amdgcn_readfirstlane((int)((uint32_t)(x >> 32) & 0xFFFFu));
    v[2] = __builtin_amdgcn_readfirstlane((int)bytes);
    v[3] = kBufferWord3;
    return v;
}
// 16 bytes per lane from rs at voff + soff into LDS at lds + 16 lane; M0 (the
// LDS destination, one wait state after writing it) is saved and restored in
// the asm
__device__ __forceinline__ void dma_b128(uint32_t lds, i4 rs, int voff, int soff)
{
    uint32_t keep;
    asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %1\n\ts_nop 0\n\t"
                 "buffer_load_dwordx4 %2, %3, %4 offen lds\n\ts_mov_b32 m0, %0"
                 : "=&s"(keep)
                 : "s"(lds), "v"(voff), "s"(rs), "s"(soff)
                 : "memory");
}
// all of this wave's loads but the N most recent, and its LDS operations, done;
// then the workgroup barrier (the waits are the compiler's own, so it counts
// them when it places its LDS waits)
template <int N> __device__ __forceinline__ void dma_barrier()
{
    __builtin_amdgcn_s_waitcnt((N & 15) | (((N >> 4) & 3) << 14) | (7 << 4));
    __builtin_amdgcn_s_barrier();
}

// acc += A_tile(128 x 64) B_tile(128 x 64)^T for this wave's 64 x 64 quarter
// (waves 2 x 2; acc[i][j] is the 16 x 16 block (i, j); lane l holds rows
// 4 (l / 16) + v, column l % 16 of it)
__device__ __forceinline__ void mma_bk(f4 (&acc)[4][4], const __bf16 *sA, const __bf16 *sB, int wm,
                                       int wn, int lane)
{
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
        bf16x8 a[4], b[4];
        const int q = ks * 4 + (lane >> 4);
#pragma unroll
        for (int i = 0; i < 4; ++i)
            a[i] = *(const bf16x8 *)(sA + lds_off(wm * 64 + i * 16 + (lane & 15), q));
#pragma unroll
        for (int j = 0; j < 4; ++j)
            b[j] = *(const bf16x8 *)(sB + lds_off(wn * 64 + j * 16 + (lane & 15), q));
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
}

// ---- bmv: y[b][k] = W[k] v[b][k] (+ bias[k]) (+ add1[b][k]) (+ add2[b][k]) -----
// for every sequence b of region k, fp32 sums of bf16 weights times fp32
// vectors; outputs y, silu(y) and silu'(y) (each optional).  A wave takes 8
// rows and 8 sequences: each weight row is read once per region and 8
// sequences, each vector chunk serves 8 rows.
struct BmvArgs {
    const __bf16 *W;
    int64_t sW;  // region stride (elements); rows N of C columns
    const float *v;
    int64_t v_sb, v_sk;
    const float *bias;
    int64_t s_bias;
    const float *add1;
    int64_t a1_sb, a1_sk;
    const float *add2;
    int64_t a2_sb, a2_sk;
    float *y, *ys, *yd;
    int64_t y_sb, y_sk;
    int64_t B;
    int N, C;
};

__global__ __launch_bounds__(kT) void bmv_kernel(BmvArgs a)
{
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int64_t k = blockIdx.y, b0 = (int64_t)blockIdx.z * 8;
    const int n0 = blockIdx.x * 32 + w * 8;
    const __bf16 *W = a.W + k * a.sW;
    float acc[64];  // [row rr][sequence bb]
#pragma unroll
    for (int i = 0; i < 64; ++i)
        acc[i] = 0.0f;
    for (int c = lane * 8; c < a.C; c += 64 * 8) {
        float v[8][8];
#pragma unroll
        for (int bb = 0; bb < 8; ++bb) {
            if (b0 + bb < a.B) {
                const float *vp = a.v + (b0 + bb) * a.v_sb + k * a.v_sk + c;
                const f4 x0 = *(const f4 *)vp, x1 = *(const f4 *)(vp + 4);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    v[bb][e] = x0[e];
                    v[bb][4 + e] = x1[e];
                }
            } else {
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    v[bb][e] = 0.0f;
            }
        }
#pragma unroll
        for (int rr = 0; rr < 8; ++rr) {
            if (n0 + rr < a.N) {
                const bf16x8 wv = *(const bf16x8 *)(W + (int64_t)(n0 + rr) * a.C + c);
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const float wf = (float)wv[e];
#pragma unroll
                    for (int bb = 0; bb < 8; ++bb)
                        acc[rr * 8 + bb] += wf * v[bb][e];
                }
            }
        }
    }
    // the 64 partial sums over the 64 lanes: lane l ends with index l
    {
        const bool upper = (lane >> 5) & 1;
#pragma unroll
        for (int i = 0; i < 32; ++i) {
            const float keep = upper ? acc[i + 32] : acc[i];
            const float send = upper ? acc[i] : acc[i + 32];
            acc[i] = keep + __shfl_xor(send, 32);
        }
        float q[32];
#pragma unroll
        for (int i = 0; i < 32; ++i)
            q[i] = acc[i];
        group_reduce<32, 32>(q, lane & 31);
        acc[0] = q[0];
    }
    const int rr = lane >> 3, bb = lane & 7;
    const int n = n0 + rr;
    const int64_t b = b0 + bb;
    if (n < a.N && b < a.B) {
        float y = acc[0];
        if (a.bias)
            y += a.bias[k * a.s_bias + n];
        if (a.add1)
            y += a.add1[b * a.a1_sb + k * a.a1_sk + n];
        if (a.add2)
            y += a.add2[b * a.a2_sb + k * a.a2_sk + n];
        const int64_t o = b * a.y_sb + k * a.y_sk + n;
        if (a.y)
            a.y[o] = y;
        if (a.ys)
            a.ys[o] = silu(y);
        if (a.yd)
            a.yd[o] = dsilu(y);
    }
}

// ---- p1: P1[k][b r + j][h] = W_d1[k][h][j] silu'(a)[b][k][h], the A operand of
//      Jdec^T; 64 values of h per workgroup, transposed through LDS so that
//      both the reads of W_d1 rows and the writes of P1 rows are contiguous
__global__ __launch_bounds__(kT) void p1_kernel(RegionArgs q)
{
    __shared__ float tile[64][129];  // [h - h0][j], r <= 128
    const int64_t bk = blockIdx.x, b = bk / q.K, k = bk % q.K;
    const int D = q.D, r = q.r;
    const int h0 = blockIdx.y * 64;
    const __bf16 *Wd1 = (const __bf16 *)q.W_d1 + k * (int64_t)D * r;
    const float *sa = q.sa + bk * D;
    for (int idx = threadIdx.x; idx < 64 * r; idx += kT) {
        const int hh = idx / r, j = idx % r;
        tile[hh][j] = bf(Wd1, (int64_t)(h0 + hh) * r + j) * sa[h0 + hh];
    }
    __syncthreads();
    __bf16 *P1 = q.P1 + (k * q.B + b) * (int64_t)r * D;
    for (int idx = threadIdx.x; idx < 64 * r; idx += kT) {
        const int j = idx / 64, hh = idx % 64;
        P1[(int64_t)j * D + h0 + hh] = (__bf16)tile[hh][j];
    }
}

// ---- xpart / xfin: mean over the tokens of x_embed, 64-token partial sums first
__global__ __launch_bounds__(kT) void xpart_kernel(RegionArgs q)
{
    // thread t sums the 8 columns 8t .. 8t + 7 over the workgroup's 64 tokens
    const int64_t b = blockIdx.y, ch = blockIdx.x;
    const int64_t l0 = ch * 64, l1 = l0 + 64 < q.L ? l0 + 64 : q.L;
    const int c = threadIdx.x * 8;
    if (c >= q.D)
        return;
    const __bf16 *x = (const __bf16 *)q.x_embed + b * q.L * q.D + c;
    float s[8] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
    // (unrolled: eight token loads in flight rather than one)
#pragma unroll 8
    for (int64_t l = l0; l < l1; ++l) {
        const bf16x8 v = *(const bf16x8 *)(x + l * q.D);
#pragma unroll
        for (int e = 0; e < 8; ++e)
            s[e] += (float)v[e];
    }
    const int64_t nch = (q.L + 63) / 64;
    float *o = q.xpart + (b * nch + ch) * q.D + c;
#pragma unroll
    for (int e = 0; e < 8; ++e)
        o[e] = s[e];
}

__global__ __launch_bounds__(kT) void xfin_kernel(RegionArgs q)
{
    const int64_t b = blockIdx.y;
    const int c = blockIdx.x * kT + threadIdx.x;
    if (c >= q.D)
        return;
    const int64_t nch = (q.L + 63) / 64;
    float s = 0.0f;
#pragma unroll 8
    for (int64_t ch = 0; ch < nch; ++ch)
        s += q.xpart[(b * nch + ch) * q.D + c];
    q.xbar[b * q.D + c] = s / (float)q.L;
}

// ---- region_dma: sbar, gbar for 128 columns of X, one sequence and region -----
// H = x_embed[b] W1[k]^T + 1 cvec[b, k]^T (cvec = W1 d) over all L tokens in
// 128-row tiles; the epilogue of each tile adds silu(H) and silu'(H) of its
// valid rows into per-lane column sums.  Both operands load straight into LDS
// (buffer_load_dwordx4 ... lds, the row layout of lds_off): 128 x 128 tiles,
// four waves of 64 x 64, two 64-deep stages (64 KB, two workgroups per CU), one
// pipeline over (row tile, k block), so that a tile's epilogue runs while the
// next tile's first stage loads.
__global__ __launch_bounds__(kT) __attribute__((amdgpu_waves_per_eu(2, 2))) void region_dma_kernel(
    RegionArgs q)
{
    constexpr int OP = BM * BK * 2;   // bytes of one operand's stage (16 KB)
    constexpr int STG = 2 * OP;
    constexpr int NL = OP / 1024 / 4; // 1 KB loads per wave, operand and stage
    __shared__ __attribute__((aligned(1024))) char smem[2 * STG];
    __shared__ float sred[2][2][BN];
    typedef __attribute__((address_space(3))) char lchar;
    const uint32_t lbase = (uint32_t)(uintptr_t)(lchar *)smem;
    const int nxt = q.X / BN;
    const int64_t G = (int64_t)gridDim.x;
    int64_t lg = blockIdx.x;
    if (G % 8 == 0)
        lg = (lg % 8) * (G / 8) + lg / 8;
    const int64_t b = lg % q.B;
    const int64_t xt = (lg / q.B) % nxt;
    const int64_t k = lg / (q.B * nxt);
    const int D = q.D;
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6), wm = w >> 1, wn = w & 1;
    const int64_t bk = b * q.K + k;
    const __bf16 *Xe = (const __bf16 *)q.x_embed + b * q.L * D;
    const i4 rsB = dma_rsrc((const __bf16 *)q.W1 + (k * q.X + xt * BN) * (int64_t)D,
                            (uint32_t)BN * D * 2);
    float cv[4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
        cv[j] = q.cvec[bk * q.X + xt * BN + wn * 64 + j * 16 + (lane & 15)];
    const int nk = D / BK;
    const int ntile = (int)((q.L + BM - 1) / BM);
    const int nstep = ntile * nk;
    // load d of a wave: rows 8 d' .. 8 d' + 7 (d' = w + 4 d) of a tile, lane ->
    // line rp = 4 d' + lane / 16, row 2 rp + (lane & 15) / 8, chunk (lane & 7) ^ (rp & 7)
    int vo[NL];
#pragma unroll
    for (int d = 0; d < NL; ++d) {
        const int rp = 4 * (w + 4 * d) + (lane >> 4);
        vo[d] = (2 * rp + ((lane & 15) >> 3)) * D * 2 + (((lane & 7) ^ (rp & 7)) << 4);
    }
    auto issue = [&](int s) {
        const int t = s / nk, kb = s - t * nk;
        const int64_t row0 = (int64_t)t * BM;
        const int vA = q.L - row0 < BM ? (int)(q.L - row0) : BM;
        const i4 rsA = dma_rsrc(Xe + row0 * D, (uint32_t)vA * D * 2);
        const uint32_t st = lbase + (uint32_t)((s & 1) * STG);
#pragma unroll
        for (int d = 0; d < NL; ++d) {
            const uint32_t blk = (uint32_t)((w + 4 * d) * 1024);
            dma_b128(__builtin_amdgcn_readfirstlane(st + blk), rsA, vo[d], kb * BK * 2);
            dma_b128(__builtin_amdgcn_readfirstlane(st + OP + blk), rsB, vo[d], kb * BK * 2);
        }
    };
    uint32_t ro[2];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
        ro[ks] = (uint32_t)(lds_off(lane & 15, 4 * ks + (lane >> 4)) * 2);
    // column sums of s = sigmoid(h), silu(h) = h s and silu(h) s
    float s1[4] = {0.0f, 0.0f, 0.0f, 0.0f}, s2[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    float s3[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    f4 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
            acc[i][j] = f4{0.0f, 0.0f, 0.0f, 0.0f};
    issue(0);
    for (int s = 0; s < nstep; ++s) {
        dma_barrier<0>();  // stage s complete; stage s - 1 read by every wave
        if (s + 1 < nstep)
            issue(s + 1);
        const uint32_t st = lbase + (uint32_t)((s & 1) * STG);
        bf16x8 a[2][4], bb[2][4];
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                a[ks][i] = *(const bf16x8 *)(lchar *)(uintptr_t)(st + ro[ks] +
                                                                  (wm * 64 + i * 16) * 128);
                bb[ks][i] = *(const bf16x8 *)(lchar *)(uintptr_t)(st + OP + ro[ks] +
                                                                   (wn * 64 + i * 16) * 128);
            }
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[ks][i], bb[ks][j],
                                                                         acc[i][j], 0, 0, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 16, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 32, 0);
        const int t = s / nk;
        if (s - t * nk == nk - 1) {
            // epilogue of row tile t over its valid rows (selects: rows past L
            // may hold anything); with s = sigmoid(h), silu = h s and
            // silu' = s + silu - silu s, the sums of s, silu and silu s carry
            // both reductions
            const int64_t rbase = (int64_t)t * BM + wm * 64 + 4 * (lane >> 4);
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const bool ok = rbase + i * 16 + v < q.L;
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const float h = acc[i][j][v] + cv[j];
                        const float sg = sigm(h);
                        const float sl = h * sg;
                        s1[j] += ok ? sg : 0.0f;
                        s2[j] += ok ? sl : 0.0f;
                        s3[j] += ok ? sl * sg : 0.0f;
                    }
                }
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    acc[i][j] = f4{0.0f, 0.0f, 0.0f, 0.0f};
        }
    }
    // lanes l, l ^ 16, l ^ 32, l ^ 48 hold the same columns; then the two
    // waves of a column half through LDS
    float cs[4], cg[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        cs[j] = s2[j];
        cg[j] = s1[j] + s2[j] - s3[j];
        cs[j] += __shfl_xor(cs[j], 16);
        cs[j] += __shfl_xor(cs[j], 32);
        cg[j] += __shfl_xor(cg[j], 16);
        cg[j] += __shfl_xor(cg[j], 32);
    }
    if (lane < 16) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            sred[0][wm][wn * 64 + j * 16 + lane] = cs[j];
            sred[1][wm][wn * 64 + j * 16 + lane] = cg[j];
        }
    }
    __syncthreads();
    if (tid < BN) {
        const float inv = 1.0f / (float)q.L;
        const int64_t o = bk * q.X + xt * BN + tid;
        q.sbar[o] = (sred[0][0][tid] + sred[0][1][tid]) * inv;
        q.gbar[o] = (sred[1][0][tid] + sred[1][1][tid]) * inv;
    }
}

// ---- ln_fwd: z = m + alpha Enc, LayerNorm -> m_{k+1}, zhat, 1/sigma ------------
__global__ __launch_bounds__(64) void ln_fwd_kernel(RegionArgs q)
{
    const int r = q.r, lane = threadIdx.x;
    const int64_t bk = blockIdx.x, k = bk % q.K;
    const float alpha = q.alpha[k];
    float z[2];
    float s = 0.0f;
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        const int i = lane + 64 * u;
        z[u] = i < r ? q.m[bk * r + i] + alpha * q.encv[bk * r + i] : 0.0f;
        s += z[u];
    }
    const float mu = wave_sum(s) / (float)r;
    float v = 0.0f;
#pragma unroll
    for (int u = 0; u < 2; ++u)
        if (lane + 64 * u < r)
            v += (z[u] - mu) * (z[u] - mu);
    const float is = 1.0f / sqrtf(wave_sum(v) / (float)r + kLnEps);
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        const int i = lane + 64 * u;
        if (i < r) {
            const float zh = (z[u] - mu) * is;
            q.zhat[bk * r + i] = zh;
            if (q.m_next)
                q.m_next[bk * r + i] = q.gamma[k * r + i] * zh + q.beta[k * r + i];
        }
    }
    if (lane == 0)
        q.isig[bk] = is;
}

// ---- gemm_nt: C[M][N] = A[M][K] B[N][K]^T per batch, with the epilogue
//      v = acc * scale[batch][row >> grp_shift][col] + add[batch][row][col] ------
struct GemmOp {
    const __bf16 *A;
    int64_t lda, sA;
    const __bf16 *B;
    int64_t ldb, sB;
    void *C;
    int64_t ldc, sC;
    int64_t M, N;
    int K;
    const float *scale;  // NULL: 1
    int64_t s_scale_b, s_scale_g;
    int grp_shift;  // rows per scale row: 2^grp_shift (1, or the interface width)
    const __bf16 *add;  // NULL: 0 (ld ldc, batch stride sC)
    bool out_bf16;
    // B's batch index is (bz0 + z) / bdiv (bdiv 0: z), so that a batch of
    // (sequence, region) pairs ordered region-major takes its region's weights
    int64_t bz0 = 0, bdiv = 0;
    // act: C = silu(v) (bf16) and C2 = silu'(v) (fp32, same index) in place of v
    bool act = false;
    float *C2 = nullptr;
};

__global__ __launch_bounds__(kT) void gemm_nt_kernel(GemmOp g)
{
    __shared__ __attribute__((aligned(16))) __bf16 sA[2][TILE];
    __shared__ __attribute__((aligned(16))) __bf16 sB[2][TILE];
    const int64_t z = blockIdx.z;
    const int64_t m0 = (int64_t)blockIdx.y * BM, n0 = (int64_t)blockIdx.x * BN;
    const __bf16 *A = g.A + z * g.sA;
    const __bf16 *B = g.B + (g.bdiv ? (g.bz0 + z) / g.bdiv : z) * g.sB;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, wm = w >> 1, wn = w & 1;
    f4 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
            acc[i][j] = f4{0.0f, 0.0f, 0.0f, 0.0f};
    const int nk = g.K / BK;
    int lkb = 0;  // next k block to load (two ahead of the products)
    uint32_t voa[4], vob[4];
    tile_offsets(voa, (int)g.lda);
    tile_offsets(vob, (int)g.ldb);
    auto load = [&](u4 (&va)[4], u4 (&vb)[4]) {
        if (lkb < nk) {
            tile_load(va, voa, A, g.lda, m0, g.M, lkb * BK);
            tile_load(vb, vob, B, g.ldb, n0, g.N, lkb * BK);
        }
        ++lkb;
    };
    u4 ra0[4], rb0[4], ra1[4], rb1[4];
    load(ra0, rb0);
    tile_store(ra0, sA[0]);
    tile_store(rb0, sB[0]);
    load(ra0, rb0);
    load(ra1, rb1);
    __syncthreads();
    int kb = 0, cur = 0;
    auto body = [&](u4 (&va)[4], u4 (&vb)[4]) -> bool {
        mma_bk(acc, sA[cur], sB[cur], wm, wn, lane);
        if (++kb == nk)
            return false;
        tile_store(va, sA[cur ^ 1]);
        tile_store(vb, sB[cur ^ 1]);
        __syncthreads();
        cur ^= 1;
        load(va, vb);
        return true;
    };
    for (;;) {
        if (!body(ra0, rb0))
            break;
        if (!body(ra1, rb1))
            break;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int64_t row = m0 + wm * 64 + i * 16 + 4 * (lane >> 4) + v;
            if (row >= g.M)
                continue;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int64_t col = n0 + wn * 64 + j * 16 + (lane & 15);
                if (col >= g.N)
                    continue;
                float val = acc[i][j][v];
                if (g.scale)
                    val *= g.scale[z * g.s_scale_b + (row >> g.grp_shift) * g.s_scale_g + col];
                const int64_t o = z * g.sC + row * g.ldc + col;
                if (g.add)
                    val += (float)g.add[o];
                if (g.act) {
                    ((__bf16 *)g.C)[o] = (__bf16)silu(val);
                    g.C2[o] = dsilu(val);
                } else if (g.out_bf16) {
                    ((__bf16 *)g.C)[o] = (__bf16)val;
                } else {
                    ((float *)g.C)[o] = val;
                }
            }
        }
}

// ---- ln_jac: J = diag(gamma) / sigma (I - 11^T/r - zhat zhat^T/r)(I + alpha Jenc),
//      stored as A[b][k] = J^T ------------------------------------------------------
__global__ __launch_bounds__(kT) void ln_jac_kernel(RegionArgs q)
{
    extern __shared__ float lsh[];
    const int r = q.r;
    float *cm = lsh;    // [r] column means of dz
    float *cd = cm + r; // [r] column dots of dz with zhat, over r
    float *zh = cd + r; // [r]
    const int64_t bk = blockIdx.x, b = bk / q.K, k = bk % q.K;
    const float alpha = q.alpha[k];
    // Jenc^T[k][b r + j][i] = Jenc[i][j]; dz = I + alpha Jenc
    const float *JT = q.JencT + (k * q.B + b) * (int64_t)r * r;
    for (int i = threadIdx.x; i < r; i += kT)
        zh[i] = q.zhat[bk * r + i];
    __syncthreads();
    for (int j = threadIdx.x; j < r; j += kT) {
        float s = 0.0f, t = 0.0f;
        for (int i = 0; i < r; ++i) {
            const float v = (i == j ? 1.0f : 0.0f) + alpha * JT[(int64_t)j * r + i];
            s += v;
            t += zh[i] * v;
        }
        cm[j] = s / (float)r;
        cd[j] = t / (float)r;
    }
    __syncthreads();
    const float is = q.isig[bk];
    float *A = q.A + bk * (int64_t)r * r;
    for (int idx = threadIdx.x; idx < r * r; idx += kT) {
        const int j = idx / r, i = idx % r;
        const float v = (i == j ? 1.0f : 0.0f) + alpha * JT[idx];
        A[idx] = q.gamma[k * r + i] * is * (v - cm[j] - zh[i] * cd[j]);
    }
}


// ==== the token-mixing block ======================================================
// Phi_k(x)_l = x_l + (W2 silu(W1 s_l)) silu(s_l) with the causal recurrence
// s_l = a_k s_{l-1} + (1 - a_k) x_l over the tokens (s_0 = 0).  The tangent of
// all r directions goes through every token: with Jdec (D x r) the same for
// each token, the state's tangent is c_l Jdec, c_l = 1 - a^l (the state of a
// constant input), and
//   dp = Jdec (1 + w) + (1/L) sum_l diag(silu(s_l)) W2 diag(silu'(W1 s_l)) W1 (c_l Jdec),
//   w  = mean_l y_l silu'(s_l) c_l,   y_l = W2 silu(W1 s_l),
// two products of r times the size of the forward's token products per
// sequence and region (Eq. "jacobian-work"), which nothing here shortcuts.

constexpr int kSsmChunks = 8;  // token chunks per channel in the recurrence kernels

// ---- ssm_fwd: s (bf16, fp32) and c for 64 channels of one pair -------------------
// Thread (channel cc, chunk ch) runs its chunk of tokens from a zero state,
// then again from the state the chunks before it leave (a chunk of n tokens
// maps a state S to a^n S + its zero-start end state).
__global__ __launch_bounds__(64 * kSsmChunks) void ssm_fwd_kernel(RegionArgs q, int64_t p0)
{
    __shared__ float endS[kSsmChunks][64], endP[kSsmChunks][64];
    const int64_t z = blockIdx.y, pr = p0 + z, k = pr / q.B, b = pr % q.B;
    const int cc = threadIdx.x & 63, ch = threadIdx.x >> 6;
    const int dch = blockIdx.x * 64 + cc;  // D is a multiple of 64
    const int D = q.D;
    const int64_t L = q.L;
    const float a = q.decay[k * D + dch];
    const float ia = 1.0f - a;
    const float dv = q.d[(b * q.K + k) * D + dch];
    const int64_t per = (L + kSsmChunks - 1) / kSsmChunks;
    const int64_t l0 = ch * per < L ? ch * per : L;
    const int64_t l1 = l0 + per < L ? l0 + per : L;
    const __bf16 *x = (const __bf16 *)q.x_embed + b * L * D + dch;
    float st = 0.0f, pw = 1.0f;
#pragma unroll 8
    for (int64_t l = l0; l < l1; ++l) {
        st = a * st + ia * ((float)x[l * D] + dv);
        pw *= a;
    }
    endS[ch][cc] = st;
    endP[ch][cc] = pw;
    __syncthreads();
    float cs = 0.0f, cc1 = 0.0f;  // states entering the chunk: of x, of the constant 1
    for (int u = 0; u < ch; ++u) {
        cs = cs * endP[u][cc] + endS[u][cc];
        cc1 = cc1 * endP[u][cc] + (1.0f - endP[u][cc]);
    }
    const int64_t o = z * L * D + dch;
#pragma unroll 8
    for (int64_t l = l0; l < l1; ++l) {
        cs = a * cs + ia * ((float)x[l * D] + dv);
        cc1 = a * cc1 + ia;
        q.s16[o + l * D] = (__bf16)cs;
        q.s32[o + l * D] = cs;
        q.c32[o + l * D] = cc1;
    }
}

// ---- ssm_red: p = mean x_embed + d + mean_l y_l silu(s_l), w = mean_l y_l silu'(s_l) c_l
__global__ __launch_bounds__(64 * kSsmChunks) void ssm_red_kernel(RegionArgs q, int64_t p0)
{
    __shared__ float r1[kSsmChunks][64], r2[kSsmChunks][64];
    const int64_t z = blockIdx.y, pr = p0 + z, k = pr / q.B, b = pr % q.B;
    const int cc = threadIdx.x & 63, ch = threadIdx.x >> 6;
    const int dch = blockIdx.x * 64 + cc;
    const int D = q.D;
    const int64_t L = q.L;
    const int64_t per = (L + kSsmChunks - 1) / kSsmChunks;
    const int64_t l0 = ch * per < L ? ch * per : L;
    const int64_t l1 = l0 + per < L ? l0 + per : L;
    const int64_t o = z * L * D + dch;
    float u1 = 0.0f, u2 = 0.0f;
#pragma unroll 8
    for (int64_t l = l0; l < l1; ++l) {
        const float y = q.y32[o + l * D], sv = q.s32[o + l * D];
        u1 = fmaf(y, silu(sv), u1);
        u2 = fmaf(y * dsilu(sv), q.c32[o + l * D], u2);
    }
    r1[ch][cc] = u1;
    r2[ch][cc] = u2;
    __syncthreads();
    if (ch == 0) {
        float t1 = 0.0f, t2 = 0.0f;
        for (int u = 0; u < kSsmChunks; ++u) {
            t1 += r1[u][cc];
            t2 += r2[u][cc];
        }
        const float inv = 1.0f / (float)L;
        const int64_t bk = b * q.K + k;
        q.p[bk * D + dch] = q.xbar[b * D + dch] + q.d[bk * D + dch] + t1 * inv;
        q.wv[z * D + dch] = t2 * inv;
    }
}

// Workgroup order of the two big tangent products: workgroup i runs on XCD
// i % 8, so logical tile lg = (i % 8) (n / 8) + i / 8 gives each XCD a
// contiguous range of logical tiles, which then share an operand in that
// XCD's L2.
__device__ __forceinline__ int64_t xcd_order(int64_t i, int64_t n)
{
    return n % 8 == 0 ? (i % 8) * (n / 8) + i / 8 : i;
}

// ---- the first tangent product: Vt[z] = (S W1[k]^T) * silu'(u)[l][x] with
//      S[l r + j][d] = c_l[d] Jdec^T[pair][j][d], stored first (ssm_s) so that
//      both operands stream straight into LDS (gen_dma below) -----------------------
struct GenArgs {
    const __bf16 *S;    // [G][L r][D]
    const __bf16 *W1;   // [K][X][D]
    const float *g32;   // [G][L][X]
    __bf16 *Vt;         // [G][L r][X]
    int64_t L, p0, Bn;
    int D, X, rs;
    int ntn, ntm;       // 256-wide column tiles, 256-row tiles of a pair
};

// ---- the second tangent product: Tpart[z][c][j][d] = sum over the tokens l of
//      256-row tile c of silu(s_l)[d] (Vt[z] W2[k]^T)[l r + j][d] ------------------
struct TokArgs {
    const __bf16 *Vt;   // [G][L r][X]
    const __bf16 *W2;   // [K][D][X]
    const float *s32;   // [G][L][D]
    float *Tpart;       // [G][nchunk][r][D], nchunk = the 256-row tiles of L r
    int64_t L, p0, Bn;  // pair z is p0 + z, of region (p0 + z) / Bn
    int X, D, r, rs, nchunk;
};

// ---- ssm_s: the first tangent product's left operand S (GenArgs above), rounded
//      to bf16 as it is formed; thread e writes the 8 values of chunk e % (D / 8)
//      of row e / (D / 8) --------------------------------------------------------------
__global__ __launch_bounds__(kT) void ssm_s_kernel(RegionArgs q, int64_t p0)
{
    const int64_t z = blockIdx.y;
    const int D = q.D, r = q.r, dq = D / 8;
    const int64_t Lr = q.L * r;
    const int64_t e = (int64_t)blockIdx.x * kT + threadIdx.x;
    if (e >= Lr * dq)
        return;
    const int64_t row = e / dq, l = row / r;
    const int c = (int)(e % dq), j = (int)(row % r);
    const float *cp = q.c32 + (z * q.L + l) * D + c * 8;
    const f4 c0 = *(const f4 *)cp, c1 = *(const f4 *)(cp + 4);
    const bf16x8 jv = *(const bf16x8 *)(q.JdT + ((p0 + z) * r + j) * D + c * 8);
    bf16x8 o;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        o[i] = (__bf16)(c0[i] * (float)jv[i]);
        o[4 + i] = (__bf16)(c1[i] * (float)jv[4 + i]);
    }
    *(bf16x8 *)(q.S16 + (z * Lr + row) * D + c * 8) = o;
}

// ==== 256 x 256 tiles with operands loaded straight into LDS ===========================
// C (256 x 256, fp32 in registers) = A rows x B rows^T over K, both bf16 with K
// contiguous.  Eight waves (2 x 4) of 128 x 64.  Two LDS stages of 64 k
// (32 KB per operand): the next stage's loads run while this stage's MFMAs
// do, one barrier per stage.  buffer_load_dwordx4 ... lds writes each lane's
// 16 bytes at M0 + 16 lane, so the operands take no registers and no VALU or
// LDS-write instructions; the rows (128 B) sit two to a 256-byte line with
// chunk q of row R in slot ((R & 1) 8 + q) ^ ((R / 2) & 7), the layout of
// lds_off, and each lane loads the global chunk that its LDS slot holds.
constexpr int kDT = 512;                  // threads
constexpr int kDOp = 256 * BK * 2;        // bytes of one operand's stage (32 KB)
constexpr int kDStage = 2 * kDOp;         // A and B
constexpr int kDLoads = kDOp / 1024 / 8;  // 1 KB loads per wave, operand and stage

// acc += the tile product over K (a multiple of 64); rows of A from rsA, of B
// from rsB (resources that end at the last valid row, so no load leaves them;
// the callers do not rely on what the products of rows past it hold)
__device__ __forceinline__ void dtile_product(f4 (&acc)[8][4], i4 rsA, i4 rsB, int K, int w,
                                              int lane, uint32_t lbase)
{
    typedef __attribute__((address_space(3))) char lchar;
    const int wm = w >> 2, wn = w & 3;
    // load d of a wave (1 KB, rows 8 d' .. 8 d' + 7 with d' = w + 8 d): lane ->
    // line rp = 4 d' + lane / 16, row 2 rp + (lane & 15) / 8, global chunk
    // (lane & 7) ^ (rp & 7)
    int vo[kDLoads];
#pragma unroll
    for (int d = 0; d < kDLoads; ++d) {
        const int rp = 4 * (w + 8 * d) + (lane >> 4);
        vo[d] = (2 * rp + ((lane & 15) >> 3)) * K * 2 + (((lane & 7) ^ (rp & 7)) << 4);
    }
    auto issue = [&](int s) {
        const uint32_t st = lbase + (uint32_t)((s & 1) * kDStage);
#pragma unroll
        for (int d = 0; d < kDLoads; ++d) {
            const uint32_t blk = (uint32_t)((w + 8 * d) * 1024);
            dma_b128(__builtin_amdgcn_readfirstlane(st + blk), rsA, vo[d], s * BK * 2);
            dma_b128(__builtin_amdgcn_readfirstlane(st + kDOp + blk), rsB, vo[d], s * BK * 2);
        }
    };
    // operand reads: row lane & 15 of a 16-row block, chunk 4 ks + lane / 16
    uint32_t ro[2];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
        ro[ks] = (uint32_t)(lds_off(lane & 15, 4 * ks + (lane >> 4)) * 2);
    const int nk = K / BK;
    issue(0);
    for (int t = 0; t < nk; ++t) {
        dma_barrier<0>();  // stage t complete; stage t - 1 read by every wave
        if (t + 1 < nk)
            issue(t + 1);
        const uint32_t st = lbase + (uint32_t)((t & 1) * kDStage);
        bf16x8 a[2][8], b[2][4];
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
#pragma unroll
            for (int i = 0; i < 8; ++i)
                a[ks][i] = *(const bf16x8 *)(lchar *)(uintptr_t)(st + ro[ks] +
                                                                  (wm * 128 + i * 16) * 128);
#pragma unroll
            for (int j = 0; j < 4; ++j)
                b[ks][j] = *(const bf16x8 *)(lchar *)(uintptr_t)(st + kDOp + ro[ks] +
                                                                  (wn * 64 + j * 16) * 128);
        }
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
#pragma unroll
            for (int i = 0; i < 8; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[ks][i], b[ks][j],
                                                                         acc[i][j], 0, 0, 0);
        // all operand reads first, then the MFMAs (each waits only for its own)
        __builtin_amdgcn_sched_group_barrier(0x100, 24, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 64, 0);
    }
}

// ---- gen_dma: the first tangent product (GenArgs above), one 256 x 256 tile of
//      one pair per workgroup; the epilogue scales by silu'(u) and stores bf16 ---
__global__ __launch_bounds__(kDT) __attribute__((amdgpu_waves_per_eu(2, 2))) void gen_dma_kernel(
    GenArgs a)
{
    __shared__ __attribute__((aligned(1024))) char smem[2 * kDStage];  // 128 KB
    typedef __attribute__((address_space(3))) char lchar;
    const uint32_t lbase = (uint32_t)(uintptr_t)(lchar *)smem;
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int64_t lg = xcd_order(blockIdx.x, (int64_t)gridDim.x);
    const int tn = (int)(lg % a.ntn);
    const int tm = (int)((lg / a.ntn) % a.ntm);
    const int64_t z = lg / ((int64_t)a.ntn * a.ntm);
    const int64_t k = (a.p0 + z) / a.Bn;
    const int64_t Lr = a.L << a.rs;
    const int64_t row0 = (int64_t)tm * 256, col0 = (int64_t)tn * 256;
    const int vA = Lr - row0 < 256 ? (int)(Lr - row0) : 256;
    const int vB = a.X - col0 < 256 ? (int)(a.X - col0) : 256;
    const int D = a.D;
    const i4 rsA = dma_rsrc(a.S + (z * Lr + row0) * D, (uint32_t)vA * D * 2);
    const i4 rsB = dma_rsrc(a.W1 + (k * a.X + col0) * D, (uint32_t)vB * D * 2);
    f4 acc[8][4];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
            acc[i][j] = f4{0.0f, 0.0f, 0.0f, 0.0f};
    dtile_product(acc, rsA, rsB, D, w, lane, lbase);
    // (a 16-row block is one token: r is a multiple of 16.)  The scale factors
    // are all loaded before the first store, so that one wait covers them.
    const int wm = w >> 2, wn = w & 3;
    const float *gz = a.g32 + z * a.L * a.X;
    __bf16 *out = a.Vt + z * Lr * a.X;
    float gs[8][4];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int64_t rb = row0 + wm * 128 + i * 16;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t col = col0 + wn * 64 + j * 16 + (lane & 15);
            gs[i][j] = rb < Lr && col < a.X ? gz[(rb >> a.rs) * a.X + col] : 0.0f;
        }
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int64_t rb = row0 + wm * 128 + i * 16;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t col = col0 + wn * 64 + j * 16 + (lane & 15);
            if (rb < Lr && col < a.X) {
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    out[(rb + 4 * (lane >> 4) + v) * a.X + col] = (__bf16)(acc[i][j][v] * gs[i][j]);
            }
        }
    }
}

// ---- tok_dma: the second tangent product (TokArgs above) on 256 x 256 tiles ------
// One workgroup: one column tile of D and one 256-row tile c of a pair (a tile
// row's token is row / r, its j is row mod r); it writes the tile's partial
// sum Tpart[z][c].  The product is weighted by silu(s_l) and summed over the
// tile's tokens: first over a wave's row blocks that share j (blocks i and
// i + NB, NB = min(r, 128) / 16), then across the tile's two row halves
// through LDS.
template <int RS>
__global__ __launch_bounds__(kDT) __attribute__((amdgpu_waves_per_eu(2, 2))) void tok_dma_kernel(
    TokArgs a)
{
    constexpr int NB = (RS >= 7 ? 128 : (1 << RS)) / 16;
    __shared__ __attribute__((aligned(1024))) char smem[2 * kDStage];  // 128 KB
    typedef __attribute__((address_space(3))) char lchar;
    const uint32_t lbase = (uint32_t)(uintptr_t)(lchar *)smem;
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6), wm = w >> 2, wn = w & 3;
    const int64_t nct = (a.D + 255) / 256;
    const int64_t lg = xcd_order(blockIdx.x, (int64_t)gridDim.x);
    const int64_t z = lg / (nct * a.nchunk);
    const int c = (int)((lg / nct) % a.nchunk);
    const int64_t col0 = (lg % nct) * 256;
    const int64_t k = (a.p0 + z) / a.Bn;
    const int64_t Lr = a.L << RS;
    const int64_t row0 = (int64_t)c * 256;
    const int vA = Lr - row0 < 256 ? (int)(Lr - row0) : 256;
    const int vB = a.D - col0 < 256 ? (int)(a.D - col0) : 256;
    const i4 rsA = dma_rsrc(a.Vt + (z * Lr + row0) * a.X, (uint32_t)vA * a.X * 2);
    const i4 rsB = dma_rsrc(a.W2 + (k * a.D + col0) * a.X, (uint32_t)vB * a.X * 2);
    f4 acc[8][4];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
            acc[i][j] = f4{0.0f, 0.0f, 0.0f, 0.0f};
    dtile_product(acc, rsA, rsB, a.X, w, lane, lbase);
    // weights, all loaded before they are used (rows past L r and columns past
    // D are left out by selects: their products may be anything)
    const float *sz = a.s32 + z * a.L * a.D;
    float wt[8][4];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int64_t l = (row0 + wm * 128 + i * 16) >> RS;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t col = col0 + wn * 64 + j * 16 + (lane & 15);
            wt[i][j] = l < a.L && col < a.D ? silu(sz[l * a.D + col]) : 0.0f;
        }
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const bool live = (row0 + wm * 128 + i * 16) < Lr;
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const float x = live ? wt[i][j] * acc[i][j][v] : 0.0f;
                if (i < NB)
                    acc[i][j][v] = x;
                else
                    acc[i % NB][j][v] += x;
            }
    }
    // the lower row half adds the upper one's sums through LDS ([j][256] fp32)
    __syncthreads();  // (every wave is past its operand reads)
    float *red = (float *)smem;
    if (wm == 1) {
#pragma unroll
        for (int i = 0; i < NB; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    red[(i * 16 + 4 * (lane >> 4) + v) * 256 + wn * 64 + j * 16 + (lane & 15)] =
                        acc[i][j][v];
    }
    __syncthreads();
    if (wm == 0) {
        float *out = a.Tpart + (z * a.nchunk + c) * ((int64_t)a.D << RS);
#pragma unroll
        for (int i = 0; i < NB; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int cl = wn * 64 + j * 16 + (lane & 15);
                if (col0 + cl < a.D) {
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        const int jr = i * 16 + 4 * (lane >> 4) + v;
                        out[(int64_t)jr * a.D + col0 + cl] = acc[i][j][v] + red[jr * 256 + cl];
                    }
                }
            }
    }
}

// ---- tfin: dp^T[pair][j][d] = Jdec^T (1 + w[d]) + (1/L) sum_c Tpart[z][c][j][d] ----
__global__ __launch_bounds__(kT) void tfin_kernel(RegionArgs q, int64_t p0)
{
    const int64_t z = blockIdx.y, pr = p0 + z;
    const int D = q.D, r = q.r;
    const int idx = blockIdx.x * kT + threadIdx.x;
    if (idx >= r * D)
        return;
    const int j = idx / D, dch = idx % D;
    // four running sums over the row tiles' partials, so that four loads are
    // in flight at a time
    const float *tp = q.Tpart + (z * q.nchunk * r + j) * (int64_t)D + dch;
    const int64_t stride = (int64_t)r * D;
    float t4[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    int c = 0;
    for (; c + 4 <= q.nchunk; c += 4) {
#pragma unroll
        for (int u = 0; u < 4; ++u)
            t4[u] += tp[(c + u) * stride];
    }
    for (; c < q.nchunk; ++c)
        t4[0] += tp[c * stride];
    const float t = (t4[0] + t4[1]) + (t4[2] + t4[3]);
    const int64_t o = (pr * r + j) * D + dch;
    q.dpT[o] = (__bf16)((float)q.JdT[o] * (1.0f + q.wv[z * D + dch]) + t / (float)q.L);
}

hipError_t gemm(const GemmOp &g, int64_t batch, hipStream_t st)
{
    const dim3 grid((unsigned)((g.N + BN - 1) / BN), (unsigned)((g.M + BM - 1) / BM),
                    (unsigned)batch);
    hipLaunchKernelGGL(gemm_nt_kernel, grid, dim3(kT), 0, st, g);
    return hipGetLastError();
}

hipError_t bmv(const BmvArgs &a, int64_t K, hipStream_t st)
{
    const dim3 grid((unsigned)((a.N + 31) / 32), (unsigned)K, (unsigned)((a.B + 7) / 8));
    hipLaunchKernelGGL(bmv_kernel, grid, dim3(kT), 0, st, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_region_jacobians(const RegionArgs &q, hipStream_t st)
{
    const int64_t BKn = q.B * q.K;
    const int64_t Br = q.B * (int64_t)q.r;
    const int D = q.D, X = q.X, r = q.r;
    const int64_t K = q.K;
    hipError_t e;
    // a = W_d1 m + b_d1 -> silu(a) (su), silu'(a) (sa)
    BmvArgs v{};
    v = BmvArgs{(const __bf16 *)q.W_d1, (int64_t)D * r, q.m, K * r, r, q.b_d1, D, nullptr, 0, 0,
                nullptr, 0, 0, nullptr, q.su, q.sa, K * D, D, q.B, D, r};
    if ((e = bmv(v, K, st)) != hipSuccess)
        return e;
    // d = W_d2 silu(a) + b_d2
    v = BmvArgs{(const __bf16 *)q.W_d2, (int64_t)D * D, q.su, K * D, D, q.b_d2, D, nullptr, 0, 0,
                nullptr, 0, 0, q.d, nullptr, nullptr, K * D, D, q.B, D, D};
    if ((e = bmv(v, K, st)) != hipSuccess)
        return e;
    hipLaunchKernelGGL(p1_kernel, dim3((unsigned)BKn, (unsigned)(D / 64)), dim3(kT), 0, st, q);
    if ((e = hipGetLastError()) != hipSuccess)
        return e;
    // cvec = W1 d
    v = BmvArgs{(const __bf16 *)q.W1, (int64_t)X * D, q.d, K * D, D, nullptr, 0, nullptr, 0, 0,
                nullptr, 0, 0, q.cvec, nullptr, nullptr, K * X, X, q.B, X, D};
    if ((e = bmv(v, K, st)) != hipSuccess)
        return e;
    hipLaunchKernelGGL(xpart_kernel, dim3((unsigned)((q.L + 63) / 64), (unsigned)q.B), dim3(kT), 0,
                       st, q);
    if ((e = hipGetLastError()) != hipSuccess)
        return e;
    hipLaunchKernelGGL(xfin_kernel, dim3((unsigned)((D + kT - 1) / kT), (unsigned)q.B), dim3(kT),
                       0, st, q);
    if ((e = hipGetLastError()) != hipSuccess)
        return e;
    hipLaunchKernelGGL(region_dma_kernel, dim3((unsigned)(K * q.B * (X / BN))), dim3(kT), 0, st,
                       q);
    if ((e = hipGetLastError()) != hipSuccess)
        return e;
    // p = W2 sbar + d + mean_l x_embed
    v = BmvArgs{(const __bf16 *)q.W2, (int64_t)D * X, q.sbar, K * X, X, nullptr, 0, q.d, K * D, D,
                q.xbar, D, 0, q.p, nullptr, nullptr, K * D, D, q.B, D, X};
    if ((e = bmv(v, K, st)) != hipSuccess)
        return e;
    // e = W_e1 p + b_e1 -> silu(e) (sue), silu'(e) (se)
    v = BmvArgs{(const __bf16 *)q.W_e1, (int64_t)D * D, q.p, K * D, D, q.b_e1, D, nullptr, 0, 0,
                nullptr, 0, 0, nullptr, q.sue, q.se, K * D, D, q.B, D, D};
    if ((e = bmv(v, K, st)) != hipSuccess)
        return e;
    // Enc = W_e2 silu(e) + b_e2
    v = BmvArgs{(const __bf16 *)q.W_e2, (int64_t)r * D, q.sue, K * D, D, q.b_e2, r, nullptr, 0, 0,
                nullptr, 0, 0, q.encv, nullptr, nullptr, K * r, r, q.B, r, D};
    if ((e = bmv(v, K, st)) != hipSuccess)
        return e;
    hipLaunchKernelGGL(ln_fwd_kernel, dim3((unsigned)BKn), dim3(64), 0, st, q);
    if ((e = hipGetLastError()) != hipSuccess)
        return e;

    const __bf16 *Wd2 = (const __bf16 *)q.W_d2, *W1 = (const __bf16 *)q.W1;
    const __bf16 *W2 = (const __bf16 *)q.W2, *We1 = (const __bf16 *)q.W_e1;
    const __bf16 *We2 = (const __bf16 *)q.W_e2;
    // the interface width is a power of two (16 .. 128): scale rows by shift
    const int rs = r == 16 ? 4 : (r == 32 ? 5 : (r == 64 ? 6 : 7));
    GemmOp g;
    // Jdec^T[k] = P1[k] W_d2[k]^T                      (B r x D, K = D)
    g = GemmOp{q.P1, D, Br * D, Wd2, D, (int64_t)D * D, q.JdT, D, Br * D, Br, D, D,
               nullptr, 0, 0, 0, nullptr, true};
    if ((e = gemm(g, q.K, st)) != hipSuccess)
        return e;
    // U'^T[k] = (Jdec^T W1[k]^T) * gbar[b][k][x]        (B r x X, K = D)
    g = GemmOp{q.JdT, D, Br * D, W1, D, (int64_t)X * D, q.UT, X, Br * X, Br, X, D,
               q.gbar, X, q.K * (int64_t)X, rs, nullptr, true};
    if ((e = gemm(g, q.K, st)) != hipSuccess)
        return e;
    // dp^T[k] = U'^T W2[k]^T + Jdec^T                   (B r x D, K = X)
    g = GemmOp{q.UT, X, Br * X, W2, X, (int64_t)D * X, q.dpT, D, Br * D, Br, D, X,
               nullptr, 0, 0, 0, q.JdT, true};
    if ((e = gemm(g, q.K, st)) != hipSuccess)
        return e;
    // T'^T[k] = (dp^T W_e1[k]^T) * silu'(e)[b][k][h]    (B r x D, K = D)
    g = GemmOp{q.dpT, D, Br * D, We1, D, (int64_t)D * D, q.TT, D, Br * D, Br, D, D,
               q.se, D, q.K * (int64_t)D, rs, nullptr, true};
    if ((e = gemm(g, q.K, st)) != hipSuccess)
        return e;
    // Jenc^T[k] = T'^T W_e2[k]^T                        (B r x r, K = D), fp32
    g = GemmOp{q.TT, D, Br * D, We2, D, (int64_t)r * D, q.JencT, r, Br * r, Br, r, D,
               nullptr, 0, 0, 0, nullptr, false};
    if ((e = gemm(g, q.K, st)) != hipSuccess)
        return e;
    hipLaunchKernelGGL(ln_jac_kernel, dim3((unsigned)BKn), dim3(kT), (size_t)3 * r * sizeof(float),
                       st, q);
    return hipGetLastError();
}

}  // namespace lbi

namespace lbi {

hipError_t launch_region_jacobians_ssm(const RegionArgs &q, hipStream_t st)
{
    const int64_t BKn = q.B * q.K;
    const int64_t Br = q.B * (int64_t)q.r;
    const int D = q.D, X = q.X, r = q.r;
    const int64_t K = q.K, L = q.L;
    const int rs = r == 16 ? 4 : (r == 32 ? 5 : (r == 64 ? 6 : 7));
    const __bf16 *Wd2 = (const __bf16 *)q.W_d2, *W1 = (const __bf16 *)q.W1;
    const __bf16 *W2 = (const __bf16 *)q.W2, *We1 = (const __bf16 *)q.W_e1;
    const __bf16 *We2 = (const __bf16 *)q.W_e2;
    hipError_t e;
    // Dec_k: a = W_d1 m + b_d1 -> silu(a), silu'(a); d = W_d2 silu(a) + b_d2
    BmvArgs v{};
    v = BmvArgs{(const __bf16 *)q.W_d1, (int64_t)D * r, q.m, K * r, r, q.b_d1, D, nullptr, 0, 0,
                nullptr, 0, 0, nullptr, q.su, q.sa, K * D, D, q.B, D, r};
    if ((e = bmv(v, K, st)) != hipSuccess)
        return e;
    v = BmvArgs{(const __bf16 *)q.W_d2, (int64_t)D * D, q.su, K * D, D, q.b_d2, D, nullptr, 0, 0,
                nullptr, 0, 0, q.d, nullptr, nullptr, K * D, D, q.B, D, D};
    if ((e = bmv(v, K, st)) != hipSuccess)
        return e;
    hipLaunchKernelGGL(p1_kernel, dim3((unsigned)BKn, (unsigned)(D / 64)), dim3(kT), 0, st, q);
    if ((e = hipGetLastError()) != hipSuccess)
        return e;
    hipLaunchKernelGGL(xpart_kernel, dim3((unsigned)((L + 63) / 64), (unsigned)q.B), dim3(kT), 0,
                       st, q);
    if ((e = hipGetLastError()) != hipSuccess)
        return e;
    hipLaunchKernelGGL(xfin_kernel, dim3((unsigned)((D + kT - 1) / kT), (unsigned)q.B), dim3(kT),
                       0, st, q);
    if ((e = hipGetLastError()) != hipSuccess)
        return e;
    GemmOp g;
    // Jdec^T[k] = P1[k] W_d2[k]^T                      (B r x D, K = D)
    g = GemmOp{q.P1, D, Br * D, Wd2, D, (int64_t)D * D, q.JdT, D, Br * D, Br, D, D,
               nullptr, 0, 0, 0, nullptr, true};
    if ((e = gemm(g, q.K, st)) != hipSuccess)
        return e;

    // the token-mixing block, G (sequence, region) pairs at a time
    const int64_t Lr = L * r;
    const int nctw = (D + 255) / 256;
    for (int64_t p0 = 0; p0 < BKn; p0 += q.G) {
        const int64_t gz = q.G < BKn - p0 ? q.G : BKn - p0;
        hipLaunchKernelGGL(ssm_fwd_kernel, dim3((unsigned)(D / 64), (unsigned)gz),
                           dim3(64 * kSsmChunks), 0, st, q, p0);
        if ((e = hipGetLastError()) != hipSuccess)
            return e;
        // silu(u), silu'(u) for u = s W1[k]^T              (L x X, K = D)
        g = GemmOp{q.s16, D, L * D, W1, D, (int64_t)X * D, q.h16, X, L * X, L, X, D,
                   nullptr, 0, 0, 0, nullptr, true, p0, q.B, true, q.g32};
        if ((e = gemm(g, gz, st)) != hipSuccess)
            return e;
        // y = silu(u) W2[k]^T                               (L x D, K = X), fp32
        g = GemmOp{q.h16, X, L * X, W2, X, (int64_t)D * X, q.y32, D, L * D, L, D, X,
                   nullptr, 0, 0, 0, nullptr, false, p0, q.B, false, nullptr};
        if ((e = gemm(g, gz, st)) != hipSuccess)
            return e;
        hipLaunchKernelGGL(ssm_red_kernel, dim3((unsigned)(D / 64), (unsigned)gz),
                           dim3(64 * kSsmChunks), 0, st, q, p0);
        if ((e = hipGetLastError()) != hipSuccess)
            return e;
        // S = c_l Jdec^T (bf16), then Vt = (S W1[k]^T) * silu'(u)[l][x]   (L r x X, K = D)
        hipLaunchKernelGGL(ssm_s_kernel, dim3((unsigned)((Lr * (D / 8) + kT - 1) / kT),
                                              (unsigned)gz),
                           dim3(kT), 0, st, q, p0);
        if ((e = hipGetLastError()) != hipSuccess)
            return e;
        const int ntn = (X + 255) / 256, ntm = (int)((Lr + 255) / 256);
        GenArgs ga{q.S16, W1, q.g32, q.Vt, L, p0, q.B, D, X, rs, ntn, ntm};
        hipLaunchKernelGGL(gen_dma_kernel, dim3((unsigned)(ntn * ntm * gz)), dim3(kDT), 0, st, ga);
        if ((e = hipGetLastError()) != hipSuccess)
            return e;
        TokArgs ta{q.Vt, W2, q.s32, q.Tpart, L, p0, q.B, X, D, r, rs, q.nchunk};
        const dim3 tgrid((unsigned)(nctw * q.nchunk * gz));
        if (rs == 4)
            hipLaunchKernelGGL(tok_dma_kernel<4>, tgrid, dim3(kDT), 0, st, ta);
        else if (rs == 5)
            hipLaunchKernelGGL(tok_dma_kernel<5>, tgrid, dim3(kDT), 0, st, ta);
        else if (rs == 6)
            hipLaunchKernelGGL(tok_dma_kernel<6>, tgrid, dim3(kDT), 0, st, ta);
        else
            hipLaunchKernelGGL(tok_dma_kernel<7>, tgrid, dim3(kDT), 0, st, ta);
        if ((e = hipGetLastError()) != hipSuccess)
            return e;
        hipLaunchKernelGGL(tfin_kernel, dim3((unsigned)((r * D + kT - 1) / kT), (unsigned)gz),
                           dim3(kT), 0, st, q, p0);
        if ((e = hipGetLastError()) != hipSuccess)
            return e;
    }

    // Enc_k and the LayerNorm, as for the token-wise block
    v = BmvArgs{(const __bf16 *)q.W_e1, (int64_t)D * D, q.p, K * D, D, q.b_e1, D, nullptr, 0, 0,
                nullptr, 0, 0, nullptr, q.sue, q.se, K * D, D, q.B, D, D};
    if ((e = bmv(v, K, st)) != hipSuccess)
        return e;
    v = BmvArgs{(const __bf16 *)q.W_e2, (int64_t)r * D, q.sue, K * D, D, q.b_e2, r, nullptr, 0, 0,
                nullptr, 0, 0, q.encv, nullptr, nullptr, K * r, r, q.B, r, D};
    if ((e = bmv(v, K, st)) != hipSuccess)
        return e;
    hipLaunchKernelGGL(ln_fwd_kernel, dim3((unsigned)BKn), dim3(64), 0, st, q);
    if ((e = hipGetLastError()) != hipSuccess)
        return e;
    g = GemmOp{q.dpT, D, Br * D, We1, D, (int64_t)D * D, q.TT, D, Br * D, Br, D, D,
               q.se, D, q.K * (int64_t)D, rs, nullptr, true};
    if ((e = gemm(g, q.K, st)) != hipSuccess)
        return e;
    g = GemmOp{q.TT, D, Br * D, We2, D, (int64_t)r * D, q.JencT, r, Br * r, Br, r, D,
               nullptr, 0, 0, 0, nullptr, false};
    if ((e = gemm(g, q.K, st)) != hipSuccess)
        return e;
    hipLaunchKernelGGL(ln_jac_kernel, dim3((unsigned)BKn), dim3(kT), (size_t)3 * r * sizeof(float),
                       st, q);
    return hipGetLastError();
}

}  // namespace lbi
