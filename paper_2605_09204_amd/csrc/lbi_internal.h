// Interfaces between the translation units of the LBI scan library (not part
// of the public C-ABI in include/lbi.h).
#ifndef LBI_INTERNAL_H
#define LBI_INTERNAL_H

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "lbi.h"

namespace lbi {

// Arithmetic of the chain kernel: fp32 storage on the fp32 matrix cores; bf16
// storage on the bf16 matrix cores (the fp32 composite fed back as hi + lo, or
// rounded once); fp32 storage as exact three-part bf16 splits on the bf16
// matrix cores.
enum : int { kF32 = 0, kBF16 = 1, kF32X = 2, kBF16R1 = 3 };

// What the chain kernel writes: every adjoint lambda_j, or every suffix
// composite (P_j, c_j) of its segment.
enum : int { kOutLambda = 0, kOutComposite = 1 };

// What the chain kernel knows of the interface widths: nothing (every tile
// R x R), the widths hint (zero-padded R x R tiles, only the blocks a slot can
// fill are read and multiplied), or the hint with compact storage (tiles at
// their true shapes back to back; kOutLambda only).
enum : int { kHintNone = 0, kHintWidths = 1, kHintCompact = 2 };

struct ScanArgs {
    const void *A;     // [B][K][R][R] storage dtype
    const void *b;     // [B][K][R] storage dtype, or NULL
    const void *lamK;  // [B][R] storage dtype (kOutLambda)
    float *lam;        // [B][K][R] (kOutLambda)
    float *Pout;       // [B][K][R][R] (kOutComposite)
    float *cout;       // [B][K][R] (kOutComposite; NULL: not written)
    int64_t K;         // slots per chain
    int64_t L;         // slots per segment; workgroup (beta, d) folds slots
                       // d*L .. min(K, (d+1)*L) - 1 into composites local to
                       // the segment (L = K: whole chains)
    int32_t S;         // segments per chain, ceil(K / L)
    int32_t agg_only;  // kOutComposite: write only each segment's aggregate
                       // (its composite at the first slot), to Pout / cout
                       // indexed [B][S] instead of [B][K]
    const float *lamSeg;  // kOutLambda with segments: lambda at the end of each
                          // segment, [B][S][R] fp32 (NULL: lamK, whole chains)
    uint32_t *progress;  // [B] or NULL (kOutLambda, whole chains): raised to the
                         // number of final adjoints after every pchunk slots
    int32_t pchunk;
    int64_t npub;        // publications per chain, ceil(K / pchunk)
    uint64_t *pub_clock;  // [B][npub] or NULL: the real-time counter at each
                          // publication (entry ceil(n / pchunk) - 1 for count n)
    // Compact (ragged) storage, hinted whole-chain kOutLambda launches only:
    // slot j of a chain holds A_j as r_j x r_{j+1} row-major, b_j and lambda_j
    // as r_j values, back to back; lambda_K as r_K values per chain.  totalA
    // and totalR are the per-chain element counts of A and of b (= lambda).
    int32_t compact;
    int32_t totalA;
    int32_t totalR;
    // The LDS-ring chain kernel: ring size in 1 KB blocks, and the row pitch
    // (elements) of zero-padded storage.
    int32_t ring;
    int32_t pitch;
    // ceil(r_k / 16) for k = 0..K as 4-bit fields, 8 per word (hinted launches)
    uint32_t wcode[(LBI_MAX_HINT_K + 1 + 7) / 8];
};

struct ChainLaunch {
    ScanArgs args;
    int64_t B;       // chains
    int32_t r;       // tile width R
    bool aff;        // b present
    bool hint;       // wcode valid
    int ncol;        // 16-column blocks of the composite that can be nonzero
    int out;         // kOutLambda or kOutComposite
    hipStream_t stream;
};

// One chain-kernel launch of grid B * S workgroups, arithmetic by file.
hipError_t launch_chain_f32(const ChainLaunch &c);
hipError_t launch_chain_f32x(const ChainLaunch &c);
hipError_t launch_chain_bf16(const ChainLaunch &c);
hipError_t launch_chain_bf16r1(const ChainLaunch &c);

// The chain scan with one wavefront per chain (bf16 storage, r <= 64, whole
// chains, kOutLambda without progress counters; a widths hint is ignored).
bool chain_wave_supported(const ChainLaunch &c);
hipError_t launch_chain_wave_bf16(const ChainLaunch &c);

// The chain scan with the A tiles streamed into an LDS ring by direct-to-LDS
// loads (bf16 storage, hi + lo arithmetic, interface widths 32/64/128 with
// r_K = 64, whole chains, kOutLambda without progress counters; c.args.ring
// and c.args.pitch set, c.args.wcode holding the widths).  maxb: blocks of
// 16 x 32 in the largest tile, 8 with storage width 64, 16 with 128.
// ring_lds_bytes: the launch's dynamic LDS.
hipError_t launch_chain_ring_bf16(const ChainLaunch &c, int maxb);
int ring_lds_bytes(int ring, bool aff);

// The chain scan with sixteen waves per chain for small batches (fp32 storage,
// split arithmetic, r = 64, whole chains, kOutLambda without progress counters
// or a widths hint).
bool chain_ksplit_supported(const ChainLaunch &c);
hipError_t launch_chain_ksplit_f32x(const ChainLaunch &c);

// The log-depth (tree) scan: one launch over chunks of tree_chunk(r) slots
// of a chain level of K slots (S = ceil(K / chunk) chunks per chain, B * S
// workgroups).  AGG: each chunk's aggregate (P [B][S][r][r], c [B][S][r]);
// otherwise every lambda of the level, each chunk from its carry (lambda at
// the start of the next chunk, lamNext [B][S][r], or lambda_K for the last).
struct TreeArgs {
    const void *A;        // [B][K][r][r], bf16 or fp32 (a_bf16 of launch_tree)
    const void *b;        // [B][K][r] in A's dtype, or NULL
    const void *lamK;     // [B][r], bf16 if lamK_bf16 else fp32
    const float *lamNext; // [B][S][r]: lambda at each chunk's start, from the
                          // level above (NULL when S = 1)
    float *lam;           // [B][K][r] out (lambda mode)
    float *Pagg;          // [B][S][r][r] out (AGG)
    float *cagg;          // [B][S][r] out (AGG), or NULL
    int64_t K;
    int32_t S;
    int32_t lamK_bf16;
};
int tree_chunk(int32_t r);
hipError_t launch_tree(const TreeArgs &a, int64_t B, int32_t r, bool a_bf16, bool aff, bool agg,
                       hipStream_t stream);

// One wave polls progress[0..B-1] (acquire, device scope) until every entry
// is at least target or max_polls polls have passed; then writes released[0]
// (1: satisfied, 0: gave up) and release_clock[0] (the real-time counter),
// either may be NULL.
hipError_t launch_wait_progress(const uint32_t *progress, int64_t B, uint32_t target,
                                int64_t max_polls, uint32_t *released, uint64_t *release_clock,
                                hipStream_t stream);

// Segment carries of the two-level scan: carry[beta][d] is lambda at the end
// of segment d (lambda_K for the last), obtained by applying the segment
// aggregates right to left; the aggregate of segment d of chain beta sits at
// index beta * cstride + d * dstride of Pa (r x r) and ca (r; NULL: no
// affine term): (K, L) when every composite was kept, (S, 1) for aggregates
// only.
hipError_t launch_carry(const float *Pa, const float *ca, const void *lamK, bool lamK_bf16,
                        float *carry, int64_t B, int32_t S, int64_t cstride, int64_t dstride,
                        int32_t r, hipStream_t stream);

// lambda_j = Pc_j carry[segment of j] + cc_j for every slot of every chain
// (every composite kept, [B][K]).
hipError_t launch_apply(const float *Pc, const float *cc, const float *carry, float *lam,
                        int64_t B, int64_t K, int64_t L, int32_t S, int32_t r,
                        hipStream_t stream);

// Spectral norm and Frobenius norm / sqrt(r) of n r x r matrices (either
// output may be NULL).
hipError_t launch_norms(const void *M, bool bf16, int64_t n, int32_t r, float *spec, float *fro,
                        hipStream_t stream);

}  // namespace lbi

#endif  // LBI_INTERNAL_H
