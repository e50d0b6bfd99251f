// Phase 1 launch arguments (host side of the region kernels), apart from the
// scan's header so that the two change independently.
#ifndef LBI_REGION_ARGS_HPP
#define LBI_REGION_ARGS_HPP

#include "lbi_internal.h"

namespace lbi {

// Phase 1 for the synthetic region map: every pointer is a device pointer;
// the workspace parts (d .. JencT) are carved by the host.
struct RegionArgs {
    // parameters, stacked over the K regions (bf16 matrices, fp32 vectors)
    const void *W_d1, *W_d2, *W1, *W2, *W_e1, *W_e2;
    const float *b_d1, *b_d2, *b_e1, *b_e2, *alpha, *gamma, *beta;
    const void *x_embed;  // [B][L][D] bf16
    const float *m;       // [B][K][r]
    float *A;             // [B][K][r][r] out: J^T
    float *m_next;        // [B][K][r] out, or NULL
    int64_t B, K, L;
    int32_t D, X, r;
    // workspace: per (b, k) vectors [B][K][n] and per-b vectors [B][n] in fp32,
    // the tangent operands [K][B r][n] in bf16
    float *su, *sa, *d, *cvec, *xpart, *xbar, *sbar, *gbar, *p, *sue, *se, *encv, *zhat, *isig,
        *JencT;
    __bf16 *P1, *JdT, *UT, *dpT, *TT;
    // the token-mixing block: per-channel decay [K][D]; (sequence, region)
    // pairs p = k B + b taken G at a time, each with its states s (bf16 and
    // fp32) and the constant-input states c [L][D], silu / silu' of W1 s
    // [L][X], y = W2 silu(W1 s) [L][D], the first tangent product's left
    // operand S [L r][D] and its scaled result Vt [L r][X], the partial sums
    // of the second over nchunk token chunks [nchunk][r][D], and w [D]
    const float *decay;
    int64_t G;
    int32_t nchunk;
    __bf16 *s16, *h16, *Vt, *S16;
    float *s32, *c32, *g32, *y32, *Tpart, *wv;
};

hipError_t launch_region_jacobians(const RegionArgs &q, hipStream_t stream);
// The same construction for the token-mixing block (q.decay set).
hipError_t launch_region_jacobians_ssm(const RegionArgs &q, hipStream_t stream);

}  // namespace lbi

#endif  // LBI_REGION_ARGS_HPP
