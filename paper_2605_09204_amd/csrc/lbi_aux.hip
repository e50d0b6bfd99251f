// Carry and apply passes of the two-level interface-adjoint scan (gfx950).
//
// The chain kernel first folds each segment of Lseg slots into its local
// suffix composites (P_j, c_j) = (A_j, b_j) o ... o (A_{e-1}, b_{e-1}), e the
// segment's end (Proposition "Scan Formulation of Backpropagation": any
// bracketing of the associative combine gives the same composites): all of
// them, or only the aggregate at the segment's first slot s_d.  Then:
//   carry: lambda at each segment end, right to left, from the aggregates:
//          lambda_{e_{S-1}} = lambda_K, lambda_{s_d} = P_{s_d} lambda_{e_d} + c_{s_d};
//   apply (when every composite was kept): lambda_j = P_j lambda_{e(j)} + c_j
//          for every slot at once (Phase 2 of Algorithm "Bounded-Interface
//          Backpropagation", with the segment's carry in place of mbar_K).
//          Otherwise the chain kernel scans each segment again from its carry.
// Both are matrix-vector work on fp32 composites: TPR lanes per row, each
// lane CPR consecutive columns (16-byte loads, coalesced across the row's
// lanes), the row sum reduced by DPP within the lane group.  The carry gives
// each chain one 256-thread workgroup and walks its S aggregates serially,
// with the loads of the next two issued ahead; the apply pass gives each
// workgroup one or more whole slots, 16 KB of composites or more.

#include "lbi_device.hpp"
#include "lbi_internal.h"

namespace lbi {
namespace {

constexpr int kThreads = 256;

template <int R> struct MatVec {
    static constexpr int TPR = kThreads / R;  // lanes per row
    static constexpr int CPR = R / TPR;       // columns per lane
    static_assert(TPR >= 2 && TPR <= 16 && (CPR % 4 == 0 || CPR == 1), "matvec geometry");
};

// Sum over this lane's CPR columns of p[e] x[col0 + e], then over the row's
// TPR lanes; every lane of the group ends with the full row sum.
template <int CPR, int TPR>
__device__ __forceinline__ float row_dot(const float (&p)[CPR], const float *x, int col0)
{
    float acc = 0.0f;
    if constexpr (CPR >= 4) {
#pragma unroll
        for (int e = 0; e < CPR; e += 4) {
            const f4 xv = *(const f4 *)&x[col0 + e];
            acc += p[e] * xv[0] + p[e + 1] * xv[1] + p[e + 2] * xv[2] + p[e + 3] * xv[3];
        }
    } else {
        acc = p[0] * x[col0];
    }
    float q[1] = {acc};
    group_reduce<TPR, 1>(q, threadIdx.x % TPR);
    return q[0];
}

// This lane's CPR consecutive columns of one row of a composite (16-byte loads).
template <int CPR>
__device__ __forceinline__ void load_row(float (&p)[CPR], const float *Prow)
{
    if constexpr (CPR >= 4) {
#pragma unroll
        for (int e = 0; e < CPR; e += 4) {
            const f4 v = *(const f4 *)&Prow[e];
            p[e] = v[0];
            p[e + 1] = v[1];
            p[e + 2] = v[2];
            p[e + 3] = v[3];
        }
    } else {
        p[0] = Prow[0];
    }
}

template <int R, bool BF16>
__global__ __launch_bounds__(kThreads) void carry_kernel(const float *Pa, const float *ca,
                                                        const void *lamK, float *carry, int32_t S,
                                                        int64_t cstride, int64_t dstride)
{
    constexpr int TPR = MatVec<R>::TPR, CPR = MatVec<R>::CPR;
    __shared__ __attribute__((aligned(16))) float sl[2][R];
    const int tid = threadIdx.x;
    const int64_t beta = blockIdx.x;
    const int row = tid / TPR, col0 = (tid % TPR) * CPR;
    const bool owner = tid % TPR == 0;
    if (tid < R) {
        const float v = BF16 ? (float)((const __bf16 *)lamK)[beta * R + tid]
                             : ((const float *)lamK)[beta * R + tid];
        sl[0][tid] = v;
        carry[(beta * S + S - 1) * R + tid] = v;
    }
    // aggregates of segments d = S-1 .. 1, prefetched two steps ahead (the
    // loads are independent of lambda; only the products wait for it)
    auto fetch = [&](int32_t d, float(&p)[CPR], float &c) {
        if (d >= 1) {
            const int64_t agg = beta * cstride + d * dstride;  // aggregate of segment d
            load_row<CPR>(p, Pa + (agg * R + row) * R + col0);
            c = ca && owner ? ca[agg * R + row] : 0.0f;
        }
    };
    int cur = 0;
    auto step = [&](int32_t d, const float(&p)[CPR], float c) {
        const float sum = row_dot<CPR, TPR>(p, sl[cur], col0);
        if (owner) {
            const float v = sum + c;
            sl[cur ^ 1][row] = v;
            carry[(beta * S + d - 1) * R + row] = v;
        }
        __syncthreads();
        cur ^= 1;
    };
    float p0[CPR], p1[CPR], p2[CPR], c0 = 0.0f, c1 = 0.0f, c2 = 0.0f;
    fetch(S - 1, p0, c0);
    fetch(S - 2, p1, c1);
    __syncthreads();
    for (int32_t d = S - 1; d >= 1; d -= 3) {
        fetch(d - 2, p2, c2);
        step(d, p0, c0);
        if (d - 1 >= 1) {
            fetch(d - 3, p0, c0);
            step(d - 1, p1, c1);
        }
        if (d - 2 >= 1) {
            fetch(d - 4, p1, c1);
            step(d - 2, p2, c2);
        }
    }
}

// The apply pass moves 16 KB of composites per workgroup or more: G slots per
// workgroup of TPR lanes per row and CPR >= 16 consecutive columns per lane.
template <int R> struct ApplyGeo {
    static constexpr int CPR = R >= 128 ? 64 : 16;
    static constexpr int TPR = R / CPR;
    static constexpr int T = R * TPR;  // lanes per slot
    static constexpr int G = kThreads / T;
    static_assert(G * T == kThreads && TPR <= 16, "apply geometry");
};

template <int R>
__global__ __launch_bounds__(kThreads) void apply_kernel(const float *Pc, const float *cc,
                                                        const float *carry, float *lam,
                                                        int64_t BK, int64_t K, int64_t Lseg,
                                                        int32_t S)
{
    using Geo = ApplyGeo<R>;
    constexpr int TPR = Geo::TPR, CPR = Geo::CPR, G = Geo::G;
    __shared__ __attribute__((aligned(16))) float sx[G][R];
    const int tid = threadIdx.x;
    const int g = tid / Geo::T, t = tid % Geo::T;
    // global slot beta * K + j of this lane group (past the end: no loads or
    // stores, but still at the barrier)
    const int64_t slot = (int64_t)blockIdx.x * G + g;
    const bool live = slot < BK;
    if (t < R && live) {
        const int64_t beta = slot / K, d = (slot % K) / Lseg;
        sx[g][t] = carry[(beta * S + d) * R + t];
    }
    __syncthreads();
    if (!live)
        return;
    const int row = t / TPR, col0 = (t % TPR) * CPR;
    float p[CPR];
    load_row<CPR>(p, Pc + (slot * R + row) * R + col0);
    const float sum = row_dot<CPR, TPR>(p, sx[g], col0);
    if (t % TPR == 0)
        lam[slot * R + row] = sum + (cc ? cc[slot * R + row] : 0.0f);
}

template <int R>
hipError_t carry_r(const float *Pa, const float *ca, const void *lamK, bool bf16, float *carry,
                   int64_t B, int32_t S, int64_t cstride, int64_t dstride, hipStream_t st)
{
    if (bf16)
        hipLaunchKernelGGL((carry_kernel<R, true>), dim3((unsigned)B), dim3(kThreads), 0, st, Pa,
                           ca, lamK, carry, S, cstride, dstride);
    else
        hipLaunchKernelGGL((carry_kernel<R, false>), dim3((unsigned)B), dim3(kThreads), 0, st, Pa,
                           ca, lamK, carry, S, cstride, dstride);
    return hipGetLastError();
}

template <int R>
hipError_t apply_r(const float *Pc, const float *cc, const float *carry, float *lam, int64_t B,
                   int64_t K, int64_t Lseg, int32_t S, hipStream_t st)
{
    constexpr int G = ApplyGeo<R>::G;
    const int64_t BK = B * K;
    hipLaunchKernelGGL((apply_kernel<R>), dim3((unsigned)((BK + G - 1) / G)), dim3(kThreads), 0,
                       st, Pc, cc, carry, lam, BK, K, Lseg, S);
    return hipGetLastError();
}


// The consumer side of the streaming scan: one wave waits until the progress
// counter of every chain has reached target.  It polls with system-scope
// acquire loads (the counters are raised with system-scope atomics, so both
// meet in memory, past every XCD's L2), with a short sleep between polls, for
// at most max_polls polls, so that the wait always ends.  The loop's exit is
// uniform across the wave (a wave-wide vote), and lane 0 records the outcome.
__global__ __launch_bounds__(64) void wait_progress_kernel(const uint32_t *progress, int64_t B,
                                                           uint32_t target, int64_t max_polls,
                                                           uint32_t *released,
                                                           uint64_t *release_clock)
{
    const int lane = (int)threadIdx.x;
    int64_t polls = 0;
    bool ok = false;
    for (;;) {
        bool mine = true;
        for (int64_t i = lane; i < B; i += 64)
            mine = mine && __hip_atomic_load(&progress[i], __ATOMIC_ACQUIRE,
                                             __HIP_MEMORY_SCOPE_SYSTEM) >= target;
        ok = __all(mine);
        if (ok || ++polls >= max_polls)
            break;
        __builtin_amdgcn_s_sleep(8);
    }
    const uint64_t t = __builtin_amdgcn_s_memrealtime();
    if (lane == 0) {
        if (released)
            released[0] = ok ? 1u : 0u;
        if (release_clock)
            release_clock[0] = t;
    }
}

}  // namespace

hipError_t launch_wait_progress(const uint32_t *progress, int64_t B, uint32_t target,
                                int64_t max_polls, uint32_t *released, uint64_t *release_clock,
                                hipStream_t stream)
{
    hipLaunchKernelGGL(wait_progress_kernel, dim3(1), dim3(64), 0, stream, progress, B, target,
                       max_polls, released, release_clock);
    return hipGetLastError();
}

hipError_t launch_carry(const float *Pa, const float *ca, const void *lamK, bool lamK_bf16,
                        float *carry, int64_t B, int32_t S, int64_t cstride, int64_t dstride,
                        int32_t r, hipStream_t stream)
{
    switch (r) {
    case 16: return carry_r<16>(Pa, ca, lamK, lamK_bf16, carry, B, S, cstride, dstride, stream);
    case 32: return carry_r<32>(Pa, ca, lamK, lamK_bf16, carry, B, S, cstride, dstride, stream);
    case 64: return carry_r<64>(Pa, ca, lamK, lamK_bf16, carry, B, S, cstride, dstride, stream);
    default: return carry_r<128>(Pa, ca, lamK, lamK_bf16, carry, B, S, cstride, dstride, stream);
    }
}

hipError_t launch_apply(const float *Pc, const float *cc, const float *carry, float *lam,
                        int64_t B, int64_t K, int64_t L, int32_t S, int32_t r, hipStream_t stream)
{
    switch (r) {
    case 16: return apply_r<16>(Pc, cc, carry, lam, B, K, L, S, stream);
    case 32: return apply_r<32>(Pc, cc, carry, lam, B, K, L, S, stream);
    case 64: return apply_r<64>(Pc, cc, carry, lam, B, K, L, S, stream);
    default: return apply_r<128>(Pc, cc, carry, lam, B, K, L, S, stream);
    }
}


}  // namespace lbi
