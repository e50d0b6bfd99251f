/*
 * lbi.h -- C-ABI of the MI355X (gfx950) interface-adjoint scan of LBI
 * ("LBI: Parallel Scan Backpropagation via Latent Bounded Interfaces").
 *
 * The operation.  A bounded-interface model joins K regions by interface
 * states m_0 .. m_K; J_k = d m_{k+1} / d m_k is the interface Jacobian
 * (Section "Implementation Details": an r_{k+1} x r_k matrix).  Theorem
 * "Bounded-Interface Backpropagation" gives the interface adjoints as
 * mbar_k = J_k^T mbar_{k+1} = (J_k^T ... J_{K-1}^T) mbar_K, and Proposition
 * "Scan Formulation of Backpropagation" computes the products by an
 * associative suffix scan.  This library adds the affine term b_k (the direct
 * gradient of any loss term that reads m_k) and returns every adjoint of
 *
 *     lambda_j = A_j lambda_{j+1} + b_j,   j = K-1 .. 0,   A_j = J_j^T,
 *
 * for B independent chains, by scanning the slots under the combine
 *
 *     (A, b) o (A', b') = (A A', A b' + b)
 *
 * (left operand = lower slot) into the suffix composites
 * (P_j, c_j) = (A_j, b_j) o ... o (A_{K-1}, b_{K-1}) and applying them:
 * lambda_j = P_j lambda_K + c_j.  With b absent this is exactly the paper's
 * Phase 2 of Algorithm "Bounded-Interface Backpropagation".
 *
 * Conventions shared by every entry point:
 *   - Pointers to tensors are DEVICE pointers on the current HIP device,
 *     allocated and owned by the caller.  The library never allocates, frees
 *     or synchronizes, and keeps no pointer after a call returns.
 *   - Calls are asynchronous: work is enqueued on `stream` (NULL = the null
 *     stream) and results are valid once the caller synchronizes it.
 *   - Argument errors are reported synchronously, before anything is
 *     enqueued, and leave every buffer untouched.  A failed launch returns
 *     LBI_ERR_HIP.  A device fault surfaces at the caller's next sync.
 *   - Layout is C-contiguous row-major; every base pointer is 16-byte aligned.
 *   - bf16 is the upper half of an IEEE binary32 (torch.bfloat16).
 *   - Non-finite inputs propagate; nothing is checked for them.
 *   - Thread-safe: no mutable global state, except the scratch array of
 *     lbi_scan_backward_noalloc (below), which its calls on one GPU share.
 */
#ifndef LBI_H
#define LBI_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* HIP stream handle (the same type as hipStream_t). */
typedef struct ihipStream_t *lbi_stream_t;

#define LBI_ABI_VERSION 12

/* Largest K for which a widths hint is used (longer chains run unhinted,
 * which gives identical results). */
#define LBI_MAX_HINT_K 2047

/* Longest chain LBI_MATH_BF16_SINGLE accepts (longer chains: LBI_ERR_SHAPE).
 * Its relative error grows like 1.2e-3 sqrt(K) (about 9.5e-3 at K = 64,
 * 1.4e-2 at K = 128 on Haar-orthogonal x diag(U[0.9, 1.1]) chains at r = 64),
 * so up to this length it stays within half the bf16 tolerance of 2e-2. */
#define LBI_BF16_SINGLE_MAX_K 64

/* Bytes of the static device scratch array of lbi_scan_backward_noalloc (one
 * per GPU the library runs on, held until the process ends). */
#define LBI_NOALLOC_SCRATCH_BYTES (64u << 20)

typedef enum {
    LBI_F32 = 0,  /* A, b, lambda_K stored as float32; float32 arithmetic   */
    LBI_BF16 = 1  /* stored as bfloat16; bf16 MFMA products, fp32 sums      */
} lbi_dtype;

/* How the products are formed (lbi_scan_backward_ex,
 * lbi_scan_suffix_products, lbi_scan_backward_streaming,
 * lbi_scan_backward_ragged).  bf16 inputs always use the bf16 matrix cores. */
typedef enum {
    LBI_MATH_DEFAULT = 0,   /* the library's choice: LBI_MATH_F32_SPLIT for
                             * fp32 at r <= 64, LBI_MATH_F32_MFMA for fp32 at
                             * r = 128; for bf16 the running fp32 composite is
                             * fed back to the matrix cores as bf16 hi + lo
                             * (two products), so the only bf16 rounding is
                             * the inputs'                                      */
    LBI_MATH_F32_MFMA = 1,  /* fp32 products on the fp32 matrix cores            */
    LBI_MATH_F32_SPLIT = 2, /* fp32 products from exact three-part bf16 splits
                             * of both operands on the bf16 matrix cores (the
                             * six partial products down to 2^-16 of the leading
                             * one), fp32 accumulation; r = 128 falls back to
                             * LBI_MATH_F32_MFMA                                 */
    LBI_MATH_BF16_SINGLE = 3 /* bf16 inputs only (else LBI_ERR_DTYPE) and
                             * K <= LBI_BF16_SINGLE_MAX_K (else
                             * LBI_ERR_SHAPE): the running composite is fed
                             * back rounded once to bf16 (one product instead
                             * of two).  Faster; each slot adds a relative
                             * rounding of up to 2^-9, and these add up like a
                             * random walk (measured about 7e-3 at K = 32 on
                             * the bf16 token-batch recipe, against 2e-6 for
                             * the default), hence the length limit.  Not
                             * taken by the wavefront-per-chain scan
                             * (LBI_ALGO_CHAIN_WAVE: LBI_ERR_DTYPE; AUTO then
                             * uses the workgroup kernel)                      */
} lbi_math;

/* How the slots of a chain are scanned (lbi_scan_backward_ex). */
typedef enum {
    LBI_ALGO_AUTO = 0,      /* for K >= 16, the one a cost model fitted to
                             * MI355X timings predicts faster: the chain scan
                             * costs K serial slot steps, the two-level scan
                             * K/S slot steps over B*S workgroups, S carry
                             * steps and 8 B K r^2 bytes of composite traffic;
                             * few long chains go two-level.  K < 16: chain.
                             * Otherwise bf16 with r <= 32 and B <= 8192 goes
                             * to LBI_ALGO_CHAIN_WAVE, and fp32 with r = 64 in
                             * the split arithmetic and B <= 256 to
                             * LBI_ALGO_CHAIN_SPLITK.  Before all of these,
                             * chains that fit one tree chunk at r <= 32
                             * (K <= 16; K >= 5 for fp32, K >= 9 for bf16;
                             * B <= 256; the default arithmetic) go to one
                             * launch of LBI_ALGO_TREE.  Where AUTO would take
                             * LBI_ALGO_CHAIN for bf16 stored at r = 128 (the
                             * default arithmetic) and the widths hint is one
                             * LBI_ALGO_CHAIN_RING takes, it takes that      */
    LBI_ALGO_CHAIN = 1,     /* one workgroup folds each whole chain right to
                             * left (K-1 combines, span K) and applies every
                             * composite to lambda_K as it forms; no workspace */
    LBI_ALGO_TWO_LEVEL = 2, /* each chain is cut into S ~ sqrt(2K) segments; a
                             * workgroup per segment folds it to its aggregate
                             * (kept in the workspace), a carry pass applies
                             * the aggregates right to left to lambda_K, and a
                             * workgroup per segment scans it again from its
                             * carry, forming every lambda_j = P_j carry + c_j
                             * (span 2K/S combines + S matrix-vector products);
                             * needs workspace, B * K < 2^31                     */
    LBI_ALGO_CHAIN_WAVE = 3 /* the chain scan with one 64-lane wavefront per
                             * chain instead of a workgroup: the same combines
                             * and apply, with A_j loaded straight into
                             * matrix-core operand registers and no barriers;
                             * for many chains (a batch of token positions).
                             * bf16 storage and r <= 64 only (else
                             * LBI_ERR_DTYPE / LBI_ERR_UNSUPPORTED_R); a widths
                             * hint is accepted and not needed; no workspace.
                             * At r <= 32 it is 1.3-1.9x faster than the
                             * workgroup kernel for B <= 4096; at r = 64 it
                             * holds two waves per SIMD and is about 10%
                             * slower.  AUTO picks it for bf16, r <= 32,
                             * B <= 8192                                       */,
    LBI_ALGO_CHAIN_SPLITK = 4 /* the chain scan with sixteen waves per chain
                             * for small batches: eight waves form the
                             * products, each product A_j P_{j+1} split over
                             * the two halves of its contraction index with
                             * the partial sums added in LDS, and eight waves
                             * stage A and store lambda.  The same arithmetic
                             * as LBI_ALGO_CHAIN with LBI_MATH_F32_SPLIT, with
                             * the sums taken in another order; one chain per
                             * CU, for batches where a slot's latency sets the
                             * time (measured 1.07-1.29x faster than
                             * LBI_ALGO_CHAIN for B <= 256, slower beyond).
                             * fp32 storage, LBI_MATH_DEFAULT or
                             * LBI_MATH_F32_SPLIT, r = 64 only (else
                             * LBI_ERR_DTYPE / LBI_ERR_UNSUPPORTED_R); a widths
                             * hint is accepted and not needed; no workspace.
                             * AUTO picks it for fp32 r = 64 in the split
                             * arithmetic with B <= 256 when it does not pick
                             * LBI_ALGO_TWO_LEVEL                              */,
    LBI_ALGO_TREE = 5       /* the log-depth scan of Proposition "Scan
                             * Formulation of Backpropagation" (span
                             * logarithmic in K, Proposition "Work-Span
                             * Decomposition"): a workgroup takes a chunk of
                             * C slots (C = 8 at r = 64, 16 at r <= 32), forms
                             * its Blelloch up-sweep of matrix products (C - 1
                             * products, log2 C deep, spread over the
                             * chunk's waves) and a vector down-sweep
                             * lambda_i = P lambda_{i+s} + c (log2 C deep);
                             * longer chains go over levels of chunk
                             * aggregates, 2L + 1 launches for K <= C^(L+1).
                             * fp32 products by the exact three-part split for
                             * both storage dtypes (LBI_MATH_DEFAULT, or
                             * LBI_MATH_F32_SPLIT; others: LBI_ERR_DTYPE);
                             * r <= 64 (else LBI_ERR_UNSUPPORTED_R); a widths
                             * hint is accepted and not needed; workspace for
                             * K > C (the aggregates and carries of each
                             * level).  For chains too few to fill the GPU    */,
    LBI_ALGO_CHAIN_RING = 6 /* the chain scan (the combines and apply of
                             * LBI_ALGO_CHAIN) with each A_j tile loaded
                             * straight from HBM into a ring of LDS blocks by
                             * buffer-to-LDS loads two slots ahead, only its
                             * live r_j x r_{j+1} part, and c_j formed on the
                             * matrix cores beside P_j: no staging registers,
                             * four chains per CU.  bf16 storage with
                             * LBI_MATH_DEFAULT or a float32 choice (else
                             * LBI_ERR_DTYPE); r in {64, 128} with every
                             * width r_k in {32, 64, 128}, r_K = 64,
                             * K <= LBI_MAX_HINT_K, and the tiles of any
                             * three consecutive slots within 36 KB of LDS
                             * (else LBI_ERR_SHAPE; no widths: every r_k = r);
                             * no workspace                                   */
} lbi_algo;

typedef enum {
    LBI_OK = 0,
    LBI_ERR_NULL = 1,          /* a required pointer is NULL                */
    LBI_ERR_SHAPE = 2,         /* B < 0, K < 1, size overflow, bad widths,  *
                                * K past LBI_BF16_SINGLE_MAX_K for         *
                                * LBI_MATH_BF16_SINGLE, widths that       *
                                * LBI_ALGO_CHAIN_RING does not take        */
    LBI_ERR_DTYPE = 3,         /* dtype not an lbi_dtype, math not an       *
                                * lbi_math, or algo not an lbi_algo         */
    LBI_ERR_UNSUPPORTED_R = 4, /* r not in {16, 32, 64, 128}                */
    LBI_ERR_WORKSPACE = 5,     /* workspace missing or too small            */
    LBI_ERR_HIP = 6,           /* the HIP runtime refused the launch        */
    LBI_ERR_ALIGN = 7,         /* a pointer is not 16-byte aligned          */
    LBI_ERR_ALIAS = 8,         /* an output (or the workspace) overlaps an  *
                                * input                                     */
    LBI_ERR_SCRATCH = 9        /* lbi_scan_backward_noalloc: the call needs *
                                * more than LBI_NOALLOC_SCRATCH_BYTES       */
} lbi_status;

/*
 * Bytes of device workspace that lbi_scan_backward (and
 * lbi_scan_backward_widths) need for (B, K, r, dt): those of the algorithm
 * LBI_ALGO_AUTO picks.  0 means the call needs none (workspace may then be
 * NULL).  Returns 0 for arguments the scan would reject.
 */
size_t lbi_scan_backward_workspace_bytes(int64_t B, int64_t K, int32_t r, lbi_dtype dt);

/*
 * As lbi_scan_backward_workspace_bytes, for a given algorithm: 0 for
 * LBI_ALGO_CHAIN, LBI_ALGO_CHAIN_WAVE, LBI_ALGO_CHAIN_SPLITK and
 * LBI_ALGO_CHAIN_RING; for
 * LBI_ALGO_TWO_LEVEL about 4 B S r (r + 2) bytes with S ~ sqrt(2K) (the
 * segment aggregates in float32, plus the carries), or 4 B K r (r + 2) while
 * every composite fits 256 MiB; for LBI_ALGO_TREE about 4 B (K / C) r (r + 2)
 * bytes summed over its levels (0 for K <= C).
 */
size_t lbi_scan_backward_workspace_bytes_ex(int64_t B, int64_t K, int32_t r, lbi_dtype dt,
                                            lbi_algo algo);

/*
 * Every interface adjoint of B independent chains.
 *
 *   A         [B][K][r][r]  A[beta][j] = J_j^T, r_j rows x r_{j+1} columns,
 *                           zero-padded to r x r; row-major.
 *   b         [B][K][r]     affine terms, or NULL for b = 0.
 *   lambda_K  [B][r]        terminal adjoints mbar_K.
 *   lambda    [B][K][r]     OUTPUT, float32 for both dtypes; slot j holds
 *                           lambda_j for j = 0..K-1 (lambda_K is the input).
 *                           Must not overlap A, b or lambda_K.
 *   B >= 0 (B = 0 is a no-op that returns LBI_OK), K >= 1,
 *   r in {16, 32, 64, 128}, dt an lbi_dtype.
 *   workspace / workspace_bytes: device scratch of at least
 *                           lbi_scan_backward_workspace_bytes(B, K, r, dt)
 *                           bytes, 16-byte aligned, not overlapping any
 *                           argument; its contents on entry do not matter.
 *   stream: the HIP stream to enqueue on.
 *
 * Precision: LBI_F32 composes and applies in float32 throughout; its matrix
 * products are formed as LBI_MATH_DEFAULT says (see lbi_scan_backward_ex).
 * LBI_BF16 multiplies bf16 operands on the matrix cores with float32
 * accumulation; the running float32 composite is fed back as a two-term bf16
 * split (hi + lo), so only the inputs are bf16-rounded.  Results are bitwise
 * reproducible run to run for a given (B, K, r, dt, math).
 */
lbi_status lbi_scan_backward(const void *A, const void *b, const void *lambda_K,
                             float *lambda, int64_t B, int64_t K, int32_t r, lbi_dtype dt,
                             void *workspace, size_t workspace_bytes, lbi_stream_t stream);

/*
 * As lbi_scan_backward, for chains whose interfaces have widths
 * r_0 .. r_K <= r (the paper's "variable-width case", Section "Scan Parallel
 * Backpropagation").  widths_host is a HOST array of K+1 entries in [1, r],
 * or NULL (then this is lbi_scan_backward).  The caller zero-pads A, b and
 * lambda_K to r; the hint only lets the kernels skip all-zero tiles, so the
 * results equal the unhinted call's.  For K > LBI_MAX_HINT_K the hint is
 * ignored.  Padded output lanes (rows >= r_j of lambda_j) are exactly 0.
 */
lbi_status lbi_scan_backward_widths(const void *A, const void *b, const void *lambda_K,
                                    float *lambda, int64_t B, int64_t K, int32_t r,
                                    lbi_dtype dt, void *workspace, size_t workspace_bytes,
                                    lbi_stream_t stream, const int32_t *widths_host);

/*
 * As lbi_scan_backward_widths (widths_host may be NULL), with the arithmetic
 * chosen by `math` and the scan by `algo`; the workspace must hold
 * lbi_scan_backward_workspace_bytes_ex(B, K, r, dt, algo) bytes (the same for
 * every `math`).  For LBI_BF16 inputs the float32 choices
 * (LBI_MATH_F32_MFMA, LBI_MATH_F32_SPLIT) act as LBI_MATH_DEFAULT, and
 * LBI_MATH_BF16_SINGLE selects the single rounding of the composite; for
 * LBI_F32 inputs LBI_MATH_BF16_SINGLE is LBI_ERR_DTYPE.  The float32 choices
 * agree to float32 rounding (they accumulate in float32 in different
 * orders); they are not bitwise equal to each other.
 */
lbi_status lbi_scan_backward_ex(const void *A, const void *b, const void *lambda_K,
                                float *lambda, int64_t B, int64_t K, int32_t r, lbi_dtype dt,
                                void *workspace, size_t workspace_bytes, lbi_stream_t stream,
                                const int32_t *widths_host, lbi_math math, lbi_algo algo);

/*
 * lbi_scan_backward_ex without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  The caller still passes the inputs and
 * the output; the two-level scan's workspace is a static device array of
 * LBI_NOALLOC_SCRATCH_BYTES (64 MiB) inside the library, one per GPU, held
 * until the process ends.  The call allocates and frees nothing.
 *
 *   A, b, lambda_K, lambda, B, K, r, dt, stream, widths_host, math, algo: as
 *   for lbi_scan_backward_ex.
 * The algorithm is the one lbi_scan_backward_ex would run.  A two-level scan
 * whose composites would not fit the array keeps only the segment aggregates
 * and scans each segment again from its carry (the form lbi_scan_backward_ex
 * takes past 256 MiB of composites); its results then agree with
 * lbi_scan_backward_ex's to float32 rounding rather than bit for bit.  A call
 * whose aggregates do not fit either returns LBI_ERR_SCRATCH before anything
 * is enqueued.  The chain algorithms use no scratch and give exactly the
 * results of lbi_scan_backward_ex.
 * Every call on one GPU uses that GPU's one array, and the array keeps the
 * last call's contents (nothing in it needs to start at zero): calls that
 * overlap on one GPU (concurrent streams, or threads) race, and must be
 * ordered by the caller.
 */
lbi_status lbi_scan_backward_noalloc(const void *A, const void *b, const void *lambda_K,
                                     float *lambda, int64_t B, int64_t K, int32_t r,
                                     lbi_dtype dt, lbi_stream_t stream,
                                     const int32_t *widths_host, lbi_math math, lbi_algo algo);

/*
 * The suffix composites themselves (Proposition "Scan Formulation of
 * Backpropagation"; Algorithm "Bounded-Interface Backpropagation", Phase 2,
 * first step): for every chain and slot j,
 *
 *     P_j = A_j A_{j+1} ... A_{K-1},   c_j = A_j c_{j+1} + b_j (c_K = 0),
 *
 * so that lambda_j = P_j lambda_K + c_j.  With b absent, P_j is the paper's
 * suffix product of interface-Jacobian transposes and c_j = 0.
 *
 *   A, b, B, K, r, dt, widths_host, math: as for lbi_scan_backward_ex.
 *   P   [B][K][r][r]  OUTPUT, float32, row-major (P_j has r_j rows and r_K
 *                     columns of the padded r x r tile; the padding is 0).
 *   c   [B][K][r]     OUTPUT, float32, or NULL (not written).  Zero when b is
 *                     NULL.
 *   P and c must not overlap A, b or each other.  No workspace.  One
 *   workgroup folds each chain with the combine code of LBI_ALGO_CHAIN.
 */
lbi_status lbi_scan_suffix_products(const void *A, const void *b, float *P, float *c, int64_t B,
                                    int64_t K, int32_t r, lbi_dtype dt, lbi_stream_t stream,
                                    const int32_t *widths_host, lbi_math math);

/*
 * lbi_scan_backward with LBI_ALGO_CHAIN, publishing progress while it runs
 * (each chain's adjoints become final in the order lambda_{K-1}, ...,
 * lambda_0), so that work on the latest regions (the region-local backward of
 * Algorithm "Bounded-Interface Backpropagation", Phase 3) can start before the
 * whole scan ends.
 *
 *   A, b, lambda_K, lambda, B, K, r, dt, stream, widths_host, math: as for
 *                   lbi_scan_backward_ex.
 *   progress [B]    uint32 in DEVICE memory, set to 0 by the caller before the
 *                   call.  progress[beta] only grows; each value n it takes
 *                   is a multiple of `chunk` or K, and by the time it is
 *                   visible (device scope, e.g. to a kernel on another stream
 *                   that reads it with acquire ordering), lambda_{K-n} ..
 *                   lambda_{K-1} of chain beta are stored and visible.  It
 *                   ends at K.
 *                   The count is raised with a system-scope atomic, so it
 *                   reaches memory as it is made (not only at the kernel's
 *                   end).  K must be below 2^32.
 *   chunk >= 1      slots per publication; each costs the chain's storing
 *                   wave a wait for its outstanding memory operations and an
 *                   L2 write-back, so larger chunks cost less (measured in
 *                   the design notes).
 *   publish_clock   [B][ceil(K / chunk)] uint64 in DEVICE memory, or NULL:
 *                   entry p of chain beta receives the GPU's constant-rate
 *                   real-time counter (s_memrealtime, 100 MHz on MI355X) when
 *                   the count (p + 1) chunk (K for the last entry) is
 *                   published; readable after the call completes.  8-byte
 *                   aligned, not overlapping any other argument.
 *
 * Results equal lbi_scan_backward_ex(..., LBI_ALGO_CHAIN) bit for bit.
 */
lbi_status lbi_scan_backward_streaming(const void *A, const void *b, const void *lambda_K,
                                       float *lambda, int64_t B, int64_t K, int32_t r,
                                       lbi_dtype dt, lbi_stream_t stream,
                                       const int32_t *widths_host, lbi_math math,
                                       uint32_t *progress, int32_t chunk,
                                       uint64_t *publish_clock);

/*
 * The consumer side of lbi_scan_backward_streaming: enqueues on `stream` a
 * wait until progress[beta] >= target for every beta < B, so that work
 * enqueued after it on that stream (the region-local backward of the latest
 * regions, Algorithm "Bounded-Interface Backpropagation", Phase 3) starts as
 * soon as lambda_{K-target} .. lambda_{K-1} of every chain are final, while
 * the scan still runs on another stream.  One wavefront polls the counters
 * (system-scope acquire loads, a short sleep between polls) and gives up
 * after max_polls polls, so the wait always ends; a poll with its sleep takes
 * on the order of a microsecond.
 *
 *   progress       [B] uint32, DEVICE memory (the streaming scan's counters).
 *   B >= 0, target any value, max_polls >= 1.
 *   released       [1] uint32 DEVICE memory, or NULL: 1 when every counter
 *                  reached target, 0 when the wait gave up.
 *   release_clock  [1] uint64 DEVICE memory, or NULL: the real-time counter
 *                  (the clock of publish_clock) when the wait ended.
 * Outputs must not overlap progress or each other.
 */
lbi_status lbi_wait_progress(const uint32_t *progress, int64_t B, uint32_t target,
                             int64_t max_polls, uint32_t *released, uint64_t *release_clock,
                             lbi_stream_t stream);

/*
 * lbi_scan_backward for interfaces of different widths, stored compactly with
 * no padding (Theorem "Bounded-Interface Backpropagation" for m_k of width r_k,
 * so that J_k is r_{k+1} x r_k and A_j = J_j^T is r_j x r_{j+1}; the paper
 * notes the variable-width case is analogous).
 *
 *   widths_host [K+1]  HOST array r_0 .. r_K, each a multiple of 16 in
 *                      16..128; 1 <= K <= LBI_MAX_HINT_K.
 *   A         per chain, A_0 .. A_{K-1} back to back, A_j as r_j rows x r_{j+1}
 *             columns row-major (dt); chain stride SA = sum_{j<K} r_j r_{j+1}.
 *   b         per chain, b_0 .. b_{K-1} back to back (r_j values each, dt);
 *             chain stride SR = sum_{j<K} r_j; or NULL (= 0).
 *   lambda_K  [B][r_K] dt.
 *   lambda    OUTPUT float32, per chain lambda_0 .. lambda_{K-1} back to back
 *             (r_j values each), chain stride SR.  Must not overlap the inputs.
 *   math      as for lbi_scan_backward_ex.
 * The chain scan (one workgroup per chain) on tiles of width R, the smallest
 * of 16, 32, 64, 128 that holds every r_k.  Results equal, bit for bit, those
 * of lbi_scan_backward_ex(..., widths, math, LBI_ALGO_CHAIN) on the same
 * values zero-padded to R x R tiles (lambda's padding rows dropped).  No
 * workspace.  Widths that break the rules give LBI_ERR_SHAPE, a NULL
 * widths_host LBI_ERR_NULL.
 */
lbi_status lbi_scan_backward_ragged(const void *A, const void *b, const void *lambda_K,
                                    float *lambda, int64_t B, int64_t K,
                                    const int32_t *widths_host, lbi_dtype dt, lbi_stream_t stream,
                                    lbi_math math);

/*
 * The interface-Jacobian statistics of the appendix "Interface Jacobian
 * Structure" (Table "jacobian-norm-final-checkpoint"): for each of n r x r
 * matrices M_i, the spectral norm ||M_i||_2 and the rank-normalised Frobenius
 * norm ||M_i||_F / sqrt(r) (the RMS singular value of a square matrix).  On
 * the A stack (A_j = J_j^T has J_j's singular values) these are the local
 * ||J_k||_2 and ||J_k||_F / sqrt(r); on the P output of
 * lbi_scan_suffix_products, the suffix ||P_k||_2.
 *
 *   M     [n][r][r]  dt storage, row-major.
 *   spec  [n]        OUTPUT float32, or NULL (not computed): ||M_i||_2, to
 *                    within 2e-5 relative.  Method: repeated normalised
 *                    squaring of M^T M on the fp32 matrix cores (24 steps),
 *                    then a Rayleigh quotient; with no spectral-gap assumption
 *                    the iteration's own error is at most r / (2 e 2^24)
 *                    relative (1.4e-6 at r = 128); the rest is float32
 *                    rounding.
 *   fro   [n]        OUTPUT float32, or NULL: ||M_i||_F / sqrt(r).
 *   n >= 0; r in {16, 32, 64, 128}.  At least one output; outputs must not
 *   overlap M or each other.  A zero matrix gives 0 in both; a matrix with a
 *   NaN or infinite entry gives NaN in both.  Zero padding of a widths-padded
 *   tile changes neither norm, but the 1/sqrt(r) factor uses the tile width.
 *   No workspace.
 */
lbi_status lbi_matrix_norms(const void *M, int64_t n, int32_t r, lbi_dtype dt, float *spec,
                            float *fro, lbi_stream_t stream);

/*
 * Phase 1 of Algorithm "Bounded-Interface Backpropagation" for a synthetic
 * region map: the interface Jacobians J_k = d m_{k+1} / d m_k, from the
 * differential applied to I_r (Eq. "jacobian-identity-construction"), of
 *
 *   m_{k+1} = LN(m_k + alpha_k Enc_k(pool(Phi_k(x_embed + Dec_k(m_k)))))
 *
 * (Eq. "concrete-region-arch") with Dec_k(m) = W_d2 silu(W_d1 m + b_d1) + b_d2,
 * Phi_k(x) = x + W2 silu(W1 x) token by token, pool = the mean over a
 * sequence's L tokens, Enc_k(p) = W_e2 silu(W_e1 p + b_e1) + b_e2, and LN a
 * LayerNorm over the r interface features (gain gamma, shift beta, eps 1e-5).
 * Every matrix of region k is the k-th of a stack; all pointers are DEVICE
 * pointers; matrices bf16, row-major [rows][cols]; vectors float32.
 */
typedef struct {
    const void *W_d1;    /* [K][D][r]  bf16 */
    const float *b_d1;   /* [K][D] */
    const void *W_d2;    /* [K][D][D]  bf16 */
    const float *b_d2;   /* [K][D] */
    const void *W1;      /* [K][X][D]  bf16 */
    const void *W2;      /* [K][D][X]  bf16 */
    const void *W_e1;    /* [K][D][D]  bf16 */
    const float *b_e1;   /* [K][D] */
    const void *W_e2;    /* [K][r][D]  bf16 */
    const float *b_e2;   /* [K][r] */
    const float *alpha;  /* [K] */
    const float *gamma;  /* [K][r] */
    const float *beta;   /* [K][r] */
} lbi_region_params;

/* Workspace bytes lbi_region_jacobians needs (0 for invalid sizes). */
size_t lbi_region_jacobians_workspace_bytes(int64_t B, int64_t K, int64_t L, int32_t D,
                                            int32_t X, int32_t r);

/*
 *   params   the K regions' parameters (HOST struct of device pointers).
 *   x_embed  [B][L][D] bf16: each sequence's token embeddings (the canvas).
 *   m        [B][K][r] float32: the interface state entering region k.
 *   A        OUTPUT [B][K][r][r] float32: A[b][k] = J_k^T at m[b][k], the
 *            operand layout of lbi_scan_backward.
 *   m_next   OUTPUT [B][K][r] float32, or NULL: R_k(m[b][k]).
 *   Sizes: B >= 0, K >= 1, L >= 1, D a multiple of 64 up to 2048, X a multiple
 *   of 128 up to 8192, r in {16, 32, 64, 128}.  Workspace of
 *   lbi_region_jacobians_workspace_bytes bytes, 256-byte aligned, owned by the
 *   caller.  Outputs must not overlap the inputs or the workspace.
 * Products run on the bf16 matrix cores with fp32 accumulation; x_embed + d
 * and the tangent intermediates are rounded to bf16 where they feed one.
 */
lbi_status lbi_region_jacobians(const lbi_region_params *params, const void *x_embed,
                                const float *m, float *A, float *m_next, int64_t B, int64_t K,
                                int64_t L, int32_t D, int32_t X, int32_t r, void *workspace,
                                size_t workspace_bytes, lbi_stream_t stream);

/*
 * Phase 1 for the same region map with a token-mixing region block, of the
 * SSM kind that the architecture section lists among the region
 * transformations: over the L tokens of a sequence,
 *
 *   s_l = a_k * s_{l-1} + (1 - a_k) * x_l   (l = 1 .. L, s_0 = 0, elementwise),
 *   Phi_k(x)_l = x_l + (W2 silu(W1 s_l)) * silu(s_l),
 *
 * with x_l = x_embed_l + Dec_k(m_k), the mean pool, Enc_k and LN as above.  The
 * tangent of all r directions is propagated through every token, as the
 * batched construction of Eq. "jacobian-identity-construction" over
 * B x L x D x r tensors does: per sequence and region, the products
 * W1 (c_l Jdec) and W2 (.) over the L r columns of the directions, whose work
 * is r times that of the token products of the forward (Eq. "jacobian-work").
 *   decay    [K][D] float32 DEVICE pointer: a_k, each in [0, 1].
 *   Other arguments, sizes, layouts and errors as lbi_region_jacobians, and
 *   additionally L r / 128 <= 65535 (else LBI_ERR_SHAPE).  The workspace
 *   (lbi_region_jacobians_ssm_workspace_bytes) holds the per-token tangent
 *   products of a group of (sequence, region) pairs at a time, up to about
 *   6 GiB plus the token-wise block's parts.
 */
size_t lbi_region_jacobians_ssm_workspace_bytes(int64_t B, int64_t K, int64_t L, int32_t D,
                                                int32_t X, int32_t r);
lbi_status lbi_region_jacobians_ssm(const lbi_region_params *params, const float *decay,
                                    const void *x_embed, const float *m, float *A, float *m_next,
                                    int64_t B, int64_t K, int64_t L, int32_t D, int32_t X,
                                    int32_t r, void *workspace, size_t workspace_bytes,
                                    lbi_stream_t stream);

/* A static, human-readable name for a status code. */
const char *lbi_status_string(lbi_status s);

/* LBI_ABI_VERSION of the built library. */
int lbi_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* LBI_H */
