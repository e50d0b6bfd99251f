// Host side of the LBI scan library: argument validation, the choice between
// the chain scan and the two-level scan, and the C-ABI of include/lbi.h.
//
// Chain scan (one launch): a workgroup folds a whole chain, K-1 combines, and
// writes every lambda_j.  Span K combines per chain; the B chains run in
// parallel.  Used when the chains alone fill the GPU.
//
// Two-level scan (three launches, workspace): the K slots of each chain are
// cut into S segments of L slots.  (1) A workgroup per segment folds it into
// its local suffix composites (K-S combines per chain in all, the same as
// the chain scan) and writes them to the workspace; (2) the carry pass
// applies the S segment aggregates right to left to lambda_K (S
// matrix-vector products per chain) to get lambda at every segment end;
// (3) the apply pass forms lambda_j = P_j carry + c_j for all slots at once.
// Span L combines + S matrix-vector products, instead of K combines.  Used
// when the chains are too few to fill the GPU.

#include <math.h>
#include <string.h>

#include <mutex>

#include "lbi_internal.h"
#include "lbi_region_args.hpp"

// ---- the static scratch array (lbi_scan_backward_noalloc) --------------------
//
// The two-level scan's workspace, for callers that cannot allocate: one array
// per GPU the library runs on, held until the process ends.  Host code never
// passes the array's name to a kernel (on the host it names a stand-in, not
// device memory): it takes the array's device address from
// hipGetSymbolAddress once per device, with that device current, and passes
// that address on.  Nothing in it needs to start at zero (the two-level scan
// writes each part before reading it), so no call clears it.
namespace lbi {
__device__ __align__(256) char scratch[LBI_NOALLOC_SCRATCH_BYTES];
}  // namespace lbi

namespace {

using namespace lbi;

constexpr size_t kScratchBytes = (size_t)LBI_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void *g_scratch_ptr[kMaxDevices];

// The scratch array's address on the current device, or NULL (with *err set)
// when the runtime does not give it.
void *scratch_address(lbi_status *err)
{
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
        *err = LBI_ERR_HIP;
        return nullptr;
    }
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch_ptr[dev]) {
        void *ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(lbi::scratch)) != hipSuccess || !ptr) {
            *err = LBI_ERR_HIP;
            return nullptr;
        }
        g_scratch_ptr[dev] = ptr;
    }
    return g_scratch_ptr[dev];
}

bool supported_r(int32_t r) { return r == 16 || r == 32 || r == 64 || r == 128; }
int waves_for_r(int32_t r) { return r == 16 ? 1 : (r == 32 ? 2 : 4); }

bool overlaps(const void *p, size_t pn, const void *q, size_t qn)
{
    if (!p || !q || pn == 0 || qn == 0)
        return false;
    const uintptr_t a = (uintptr_t)p, b = (uintptr_t)q;
    return a < b + qn && b < a + pn;
}

bool misaligned(const void *p) { return p && ((uintptr_t)p & 15u); }

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Segments of the two-level scan: S ~ sqrt(2K) balances the K/S slot steps of
// a segment pass (each a chain-kernel slot step, plus a pipeline start per
// workgroup) against the S carry steps; a sweep over S on MI355X (B = 1..128,
// K = 128..2048, r = 64) puts the optimum there, within 5% or a flat region.
// Two forms:
//   * every composite kept (fp32, 4 B K r^2 bytes written and read again),
//     then one parallel apply pass: the shorter span, for small batches;
//   * aggregates only, then each segment scanned again from its carry: the
//     composites never reach memory (A is read twice instead), for batches
//     whose composites would not fit the 256 MB last-level cache.  Measured
//     at r = 64 fp32, K = 512, same box: 2% slower at B = 16 (134 MB of
//     composites), 14% faster at B = 64 (537 MB), 33% slower at B = 1.
constexpr double kRescanBytes = 256.0 * (1 << 20);

struct TwoLevelPlan {
    int64_t L;
    int32_t S;
    bool rescan;
    size_t offP, offc, offcarry, bytes;
};

// (force_rescan: the aggregates-only form whatever the composites' size)
TwoLevelPlan two_level_plan(int64_t B, int64_t K, int32_t r, bool force_rescan = false)
{
    TwoLevelPlan p;
    int64_t S = (int64_t)ceil(sqrt(2.0 * (double)K));
    if (S > K)
        S = K;
    if (S < 1)
        S = 1;
    p.L = (K + S - 1) / S;
    p.S = (int32_t)((K + p.L - 1) / p.L);
    p.rescan = force_rescan || 4.0 * (double)B * K * r * r > kRescanBytes;
    const int64_t nslots = p.rescan ? (int64_t)p.S : K;  // composites kept per chain
    const size_t nP = (size_t)B * nslots * r * r * sizeof(float);
    const size_t nc = (size_t)B * nslots * r * sizeof(float);
    const size_t ncar = (size_t)B * p.S * r * sizeof(float);
    p.offP = 0;
    p.offc = align256(nP);
    p.offcarry = p.offc + align256(nc);
    p.bytes = p.offcarry + align256(ncar);
    return p;
}

// The apply pass launches up to B*K workgroups.
bool two_level_possible(int64_t B, int64_t K) { return B * K < ((int64_t)1 << 31) - 1; }

// The tree scan over levels: level 0 is the chain of K slots, level l + 1
// the chain of the chunk aggregates of level l (len[l + 1] = ceil(len[l] /
// chunk)), up to the first level that fits one chunk.  Workspace per level
// l >= 1: the aggregates P [B][len][r][r] and c [B][len][r] (with b), and the
// lambda at each element's start [B][len][r], each 256-byte aligned.
constexpr int kMaxTreeLevels = 24;
struct TreePlan {
    int nlev;  // levels above the slots
    int64_t len[kMaxTreeLevels + 1];
    size_t offP[kMaxTreeLevels + 1], offc[kMaxTreeLevels + 1], offl[kMaxTreeLevels + 1];
    size_t bytes;
};

TreePlan tree_plan(int64_t B, int64_t K, int32_t r, bool aff)
{
    TreePlan t;
    const int64_t C = tree_chunk(r);
    t.nlev = 0;
    t.len[0] = K;
    while (t.len[t.nlev] > C && t.nlev < kMaxTreeLevels) {
        t.len[t.nlev + 1] = (t.len[t.nlev] + C - 1) / C;
        ++t.nlev;
    }
    size_t o = 0;
    for (int l = 1; l <= t.nlev; ++l) {
        t.offP[l] = o;
        o += align256((size_t)B * t.len[l] * r * r * sizeof(float));
        t.offc[l] = o;
        if (aff)
            o += align256((size_t)B * t.len[l] * r * sizeof(float));
        t.offl[l] = o;
        o += align256((size_t)B * t.len[l] * r * sizeof(float));
    }
    t.bytes = o;
    return t;
}

// The tree scan launches up to B * ceil(K / chunk) workgroups.
bool tree_possible(int64_t B, int64_t K, int32_t r)
{
    const int64_t C = tree_chunk(r);
    return B * ((K + C - 1) / C) < ((int64_t)1 << 31) - 1;
}

// Every launch of the tree scan (see the level plan above).
hipError_t run_tree(const void *A, const void *b, const void *lamK, float *lam, int64_t B,
                    int64_t K, int32_t r, lbi_dtype dt, void *ws, hipStream_t st)
{
    const bool aff = b != nullptr, bf = dt == LBI_BF16;
    const TreePlan t = tree_plan(B, K, r, aff);
    char *w = (char *)ws;
    auto Pl = [&](int l) { return (float *)(w + t.offP[l]); };
    auto cl = [&](int l) { return aff ? (float *)(w + t.offc[l]) : nullptr; };
    auto ll = [&](int l) { return (float *)(w + t.offl[l]); };
    auto level_in = [&](int l, TreeArgs &a) {
        a.A = l == 0 ? A : (const void *)Pl(l);
        a.b = l == 0 ? b : (const void *)cl(l);
        a.K = t.len[l];
    };
    TreeArgs a;
    // up: each level's chunk aggregates
    for (int l = 0; l < t.nlev; ++l) {
        memset(&a, 0, sizeof a);
        level_in(l, a);
        a.S = (int32_t)t.len[l + 1];
        a.Pagg = Pl(l + 1);
        a.cagg = cl(l + 1);
        const hipError_t e = launch_tree(a, B, r, l == 0 && bf, aff, true, st);
        if (e != hipSuccess)
            return e;
    }
    // down: the top level from lambda_K, then each level from the carries of
    // the level above
    for (int l = t.nlev; l >= 0; --l) {
        memset(&a, 0, sizeof a);
        level_in(l, a);
        a.S = l == t.nlev ? 1 : (int32_t)t.len[l + 1];
        a.lamNext = l == t.nlev ? nullptr : ll(l + 1);
        a.lamK = lamK;
        a.lamK_bf16 = bf ? 1 : 0;
        a.lam = l == 0 ? lam : ll(l);
        const hipError_t e = launch_tree(a, B, r, l == 0 && bf, aff, false, st);
        if (e != hipSuccess)
            return e;
    }
    return hipSuccess;
}

// Microseconds per slot of one chain-kernel workgroup on an otherwise idle
// MI355X (r = 16, 32, 64, 128; fp32 storage in the default arithmetic).
double slot_us(lbi_dtype dt, int32_t r)
{
    const int i = r == 16 ? 0 : (r == 32 ? 1 : (r == 64 ? 2 : 3));
    static const double f32[4] = {0.44, 0.72, 1.42, 8.67}, bf16[4] = {0.40, 0.62, 0.95, 2.91};
    return dt == LBI_BF16 ? bf16[i] : f32[i];
}

// Chains per launch up to which AUTO takes LBI_ALGO_CHAIN_SPLITK: one per CU.
constexpr int64_t kSplitKMaxB = 256;
// Chains per launch up to which AUTO takes a single launch of LBI_ALGO_TREE
// (the batches it was measured on).
constexpr int64_t kTreeMaxB = 256;

// LBI_ALGO_AUTO: the cheaper of the two by a cost model fitted to MI355X
// timings (B = 1..512, K = 32..512, every r; within 13% of the faster choice
// everywhere on that grid).  Chain scan: K serial slot steps, slower once the
// chains hold more than 1280 waves.  Two-level scan: K/S slot steps over B*S
// workgroups, S carry steps, and the composites written and read once
// (8 B K r^2 bytes at 5.8 TB/s).
// Chains that the two-level scan does not take: bf16 chains of width <= 32
// go to the wavefront-per-chain kernel (no barrier, no LDS staging), which
// measured 1.3-1.9x faster than the workgroup kernel up to B = 4096 and no
// slower up to 8192; at r = 64 its registers allow two waves per SIMD and the
// workgroup kernel is faster.  fp32 chains at r = 64 in the split arithmetic,
// at most one per CU, go to the sixteen-wave kernel (split contraction,
// specialised staging waves): 1.2-1.3x faster than the workgroup kernel for
// B <= 128 and 1.07-1.2x at B = 256, and slower once chains share CUs.  The choice between the
// chain and two-level scans does not depend on the arithmetic, so the
// workspace query needs none.
lbi_algo resolve_algo(lbi_algo algo, int64_t B, int64_t K, int32_t r, lbi_dtype dt, lbi_math math)
{
    if (algo != LBI_ALGO_AUTO)
        return algo;
    // one launch of the tree scan (K within a chunk) at r <= 32: kernel
    // times on MI355X (rocprofv3, B = 1..256) put it ahead of the chain
    // kernels there, about twice as fast for fp32 at K = 16 (6.4 against
    // 12.7 us at r = 32), for bf16 only past K = 8 (at smaller K the
    // wavefront-per-chain kernel is as fast or faster); at r = 64 the chain
    // kernels win
    if (r <= 32 && B <= kTreeMaxB && K <= tree_chunk(r) && math != LBI_MATH_F32_MFMA &&
        math != LBI_MATH_BF16_SINGLE && K >= (dt == LBI_F32 ? 5 : 9))
        return LBI_ALGO_TREE;
    const lbi_algo chain =
        dt == LBI_BF16 && math != LBI_MATH_BF16_SINGLE && r <= 32 && B <= 8192 ? LBI_ALGO_CHAIN_WAVE
        : dt == LBI_F32 && math != LBI_MATH_F32_MFMA && r == 64 && B <= kSplitKMaxB
            ? LBI_ALGO_CHAIN_SPLITK
            : LBI_ALGO_CHAIN;
    if (K < 16 || !two_level_possible(B, K))
        return chain;
    const double ts = slot_us(dt, r), w = waves_for_r(r), cap = 1280.0;
    const double t_chain = 6.0 + (double)K * ts * fmax(1.0, (double)B * w / cap);
    const TwoLevelPlan p = two_level_plan(B, K, r);
    // (three launches: 18 us of fixed cost, measured with HIP events at
    // B = 1..16, K = 16..64, where the chain scan's one launch costs 6 us
    // plus its slots)
    const double two = 18.0 + (double)p.L * ts * fmax(1.0, (double)B * p.S * w / cap) +
                       0.22 * p.S * sqrt(r / 64.0) + 8.0 * (double)B * K * r * r / 5.8e6;
    return two < t_chain ? LBI_ALGO_TWO_LEVEL : chain;
}

bool valid_algo(lbi_algo algo)
{
    return algo == LBI_ALGO_AUTO || algo == LBI_ALGO_CHAIN || algo == LBI_ALGO_TWO_LEVEL ||
           algo == LBI_ALGO_CHAIN_WAVE || algo == LBI_ALGO_CHAIN_SPLITK || algo == LBI_ALGO_TREE ||
           algo == LBI_ALGO_CHAIN_RING;
}

// The LDS-ring chain kernel (lbi_chain_ring.hip).  Shapes it takes: storage
// width r of 64 or 128, every interface width 32, 64 or 128 (at most r),
// r_K = 64, K within the widths hint.  A tile of slot j is
// (r_j / 16) x (r_{j+1} / 32) blocks of 1 KB; the kernel keeps the tiles of
// three consecutive slots in a ring of blocks, each placed right after the
// previous one, or at block 0 when it would pass the ring's end.  The ring
// size is the smallest, from the largest three-slot sum up, for which that
// rule never overlaps three consecutive tiles (the rule is run here, the same
// way); at most kRingMaxBlocks, so that four chains share a CU.
constexpr int kRingMaxBlocks = 36;
struct RingPlan {
    bool ok;
    int ring, maxb;
};
RingPlan ring_plan(const int32_t *widths, int64_t K, int32_t r)
{
    RingPlan p{false, 0, 0};
    if ((r != 64 && r != 128) || K < 1 || K > LBI_MAX_HINT_K)
        return p;
    auto wd = [&](int64_t k) { return widths ? widths[k] : r; };
    for (int64_t k = 0; k <= K; ++k) {
        const int32_t x = wd(k);
        if ((x != 32 && x != 64 && x != 128) || x > r)
            return p;
    }
    if (wd(K) != 64)
        return p;
    auto blocks = [&](int64_t j) { return j >= 0 ? (wd(j) / 16) * (wd(j + 1) / 32) : 0; };
    int win = 0;
    for (int64_t j = 0; j < K; ++j) {
        if (blocks(j) > (r == 64 ? 8 : 16))
            return p;
        const int s3 = blocks(j) + blocks(j - 1) + blocks(j - 2);
        win = s3 > win ? s3 : win;
    }
    for (int ring = win; ring <= kRingMaxBlocks; ++ring) {
        // bases of tiles K-1, K-2, ... by the kernel's rule; tiles j, j-1,
        // j-2 must not overlap (each sits inside the ring by construction)
        int b0 = 0, b1 = -1, b2 = -1;  // bases of tiles j, j+1, j+2
        bool good = true;
        for (int64_t j = K - 1; j >= 0 && good; --j) {
            if (j < K - 1) {
                const int nxt = b1 + blocks(j + 1);
                b0 = nxt + blocks(j) <= ring ? nxt : 0;
            }
            auto disjoint = [&](int ba, int64_t ja, int bb, int64_t jb) {
                return ba + blocks(ja) <= bb || bb + blocks(jb) <= ba;
            };
            if (j + 1 <= K - 1 && !disjoint(b0, j, b1, j + 1))
                good = false;
            if (j + 2 <= K - 1 && !disjoint(b0, j, b2, j + 2))
                good = false;
            b2 = b1;
            b1 = b0;
        }
        if (good) {
            p.ok = true;
            p.ring = ring;
            p.maxb = r == 64 ? 8 : 16;
            return p;
        }
    }
    return p;
}

lbi_status check_common(lbi_dtype dt, lbi_math math, int32_t r, int64_t B, int64_t K)
{
    if (dt != LBI_F32 && dt != LBI_BF16)
        return LBI_ERR_DTYPE;
    if (math != LBI_MATH_DEFAULT && math != LBI_MATH_F32_MFMA && math != LBI_MATH_F32_SPLIT &&
        math != LBI_MATH_BF16_SINGLE)
        return LBI_ERR_DTYPE;
    if (math == LBI_MATH_BF16_SINGLE && dt != LBI_BF16)
        return LBI_ERR_DTYPE;
    if (!supported_r(r))
        return LBI_ERR_UNSUPPORTED_R;
    if (B < 0 || K < 1)
        return LBI_ERR_SHAPE;
    // the single rounding's error grows like sqrt(K): only chains short
    // enough to stay within half the bf16 tolerance
    if (math == LBI_MATH_BF16_SINGLE && K > LBI_BF16_SINGLE_MAX_K)
        return LBI_ERR_SHAPE;
    // sizes must fit comfortably in 64 bits and the launch grid
    const int64_t kMax = (int64_t)1 << 40;
    if (B > (int64_t)INT32_MAX || K > kMax / ((int64_t)r * r) || B > kMax / (K * (int64_t)r * r))
        return LBI_ERR_SHAPE;
    return LBI_OK;
}

// Fills the widths code of a launch; false for widths out of range.
bool encode_widths(const int32_t *widths, int64_t K, int32_t r, ChainLaunch &c)
{
    c.hint = false;
    c.ncol = r / 16;
    if (!widths)
        return true;
    for (int64_t k = 0; k <= K; ++k)
        if (widths[k] < 1 || widths[k] > r)
            return false;
    if (K <= LBI_MAX_HINT_K) {
        c.hint = true;
        for (int64_t k = 0; k <= K; ++k) {
            const uint32_t code = (uint32_t)(widths[k] + 15) / 16;
            c.args.wcode[k >> 3] |= code << ((k & 7) * 4);
        }
        c.ncol = (widths[K] + 15) / 16;
    }
    return true;
}

hipError_t launch_chain_mode(const ChainLaunch &c, lbi_dtype dt, lbi_math math)
{
    if (dt == LBI_BF16)
        return math == LBI_MATH_BF16_SINGLE ? launch_chain_bf16r1(c) : launch_chain_bf16(c);
    if (math == LBI_MATH_F32_MFMA || c.r == 128)
        return launch_chain_f32(c);
    return launch_chain_f32x(c);
}

// With scratch = true, ws / ws_bytes are the library's static scratch array:
// a two-level scan whose composites do not fit it takes the aggregates-only
// form, and one that does not fit even so is LBI_ERR_SCRATCH.
lbi_status scan_impl(const void *A, const void *b, const void *lamK, float *lam, int64_t B,
                     int64_t K, int32_t r, lbi_dtype dt, void *ws, size_t ws_bytes,
                     lbi_stream_t stream, const int32_t *widths, lbi_math math, lbi_algo algo,
                     bool scratch = false)
{
    lbi_status st = check_common(dt, math, r, B, K);
    if (st != LBI_OK)
        return st;
    if (!valid_algo(algo))
        return LBI_ERR_DTYPE;
    if (algo == LBI_ALGO_TWO_LEVEL && !two_level_possible(B, K))
        return LBI_ERR_SHAPE;
    // the tree scan: the split arithmetic for fp32 (the default), r <= 64
    if (algo == LBI_ALGO_TREE && (math == LBI_MATH_F32_MFMA || math == LBI_MATH_BF16_SINGLE))
        return LBI_ERR_DTYPE;
    if (algo == LBI_ALGO_TREE && r > 64)
        return LBI_ERR_UNSUPPORTED_R;
    if (algo == LBI_ALGO_TREE && !tree_possible(B, K, r))
        return LBI_ERR_SHAPE;
    if (algo == LBI_ALGO_CHAIN_WAVE && (dt != LBI_BF16 || math == LBI_MATH_BF16_SINGLE))
        return LBI_ERR_DTYPE;
    if (algo == LBI_ALGO_CHAIN_WAVE && r > 64)
        return LBI_ERR_UNSUPPORTED_R;
    if (algo == LBI_ALGO_CHAIN_SPLITK && (dt != LBI_F32 || math == LBI_MATH_F32_MFMA))
        return LBI_ERR_DTYPE;
    if (algo == LBI_ALGO_CHAIN_SPLITK && r != 64)
        return LBI_ERR_UNSUPPORTED_R;
    if (algo == LBI_ALGO_CHAIN_RING && (dt != LBI_BF16 || math == LBI_MATH_BF16_SINGLE))
        return LBI_ERR_DTYPE;
    if (algo == LBI_ALGO_CHAIN_RING && !ring_plan(widths, K, r).ok)
        return LBI_ERR_SHAPE;
    if (B == 0)
        return LBI_OK;
    if (!A || !lamK || !lam)
        return LBI_ERR_NULL;
    if (misaligned(A) || misaligned(b) || misaligned(lamK) || misaligned(lam) || misaligned(ws))
        return LBI_ERR_ALIGN;
    const size_t esz = dt == LBI_F32 ? 4 : 2;
    const size_t nA = (size_t)B * K * r * r * esz, nb = b ? (size_t)B * K * r * esz : 0;
    const size_t nl = (size_t)B * r * esz, nout = (size_t)B * K * r * sizeof(float);
    if (overlaps(lam, nout, A, nA) || overlaps(lam, nout, b, nb) || overlaps(lam, nout, lamK, nl))
        return LBI_ERR_ALIAS;
    lbi_algo use = resolve_algo(algo, B, K, r, dt, math);
    // bf16 chains stored at width 128 whose widths the LDS-ring kernel takes
    // (the mixed-width case): that kernel, measured 1.45x faster there than
    // the workgroup kernel (188 against 275 us on 1024 chains of 64 slots of
    // widths 32/64/128); at width 64 the two tie
    if (algo == LBI_ALGO_AUTO && use == LBI_ALGO_CHAIN && dt == LBI_BF16 &&
        math != LBI_MATH_BF16_SINGLE && r == 128 && ring_plan(widths, K, r).ok)
        use = LBI_ALGO_CHAIN_RING;
    TwoLevelPlan p = two_level_plan(B, K, r);
    size_t need = lbi_scan_backward_workspace_bytes_ex(B, K, r, dt, use);
    if (scratch && need > kScratchBytes) {
        if (use == LBI_ALGO_TWO_LEVEL) {
            p = two_level_plan(B, K, r, true);
            need = p.bytes;
        }
        if (need > kScratchBytes)
            return LBI_ERR_SCRATCH;
    }
    if (scratch && need > 0) {
        // the library's own array: distinct from every caller buffer
        lbi_status err = LBI_OK;
        ws = scratch_address(&err);
        if (!ws)
            return err;
        ws_bytes = kScratchBytes;
    } else {
        if (need > 0 && (!ws || ws_bytes < need))
            return LBI_ERR_WORKSPACE;
        if (need > 0 && (overlaps(ws, need, A, nA) || overlaps(ws, need, b, nb) ||
                         overlaps(ws, need, lamK, nl) || overlaps(ws, need, lam, nout)))
            return LBI_ERR_ALIAS;
    }

    ChainLaunch c;
    memset(&c, 0, sizeof c);
    c.args.A = A;
    c.args.b = b;
    c.args.lamK = lamK;
    c.args.K = K;
    c.B = B;
    c.r = r;
    c.aff = b != nullptr;
    c.stream = (hipStream_t)stream;
    if (!encode_widths(widths, K, r, c))
        return LBI_ERR_SHAPE;

    if (use == LBI_ALGO_TREE)
        return run_tree(A, b, lamK, lam, B, K, r, dt, ws, c.stream) == hipSuccess ? LBI_OK
                                                                                  : LBI_ERR_HIP;
    if (use == LBI_ALGO_CHAIN_RING) {
        const RingPlan rp = ring_plan(widths, K, r);
        c.args.lam = lam;
        c.args.L = K;
        c.args.S = 1;
        c.args.ring = rp.ring;
        c.args.pitch = r;
        c.out = kOutLambda;
        if (!c.hint) {
            // uniform widths: the kernel reads them from the width codes
            const int32_t code = r / 16;
            for (int64_t k = 0; k <= K; ++k)
                c.args.wcode[k >> 3] |= (uint32_t)code << ((k & 7) * 4);
        }
        return launch_chain_ring_bf16(c, rp.maxb) == hipSuccess ? LBI_OK : LBI_ERR_HIP;
    }
    if (use == LBI_ALGO_CHAIN || use == LBI_ALGO_CHAIN_WAVE || use == LBI_ALGO_CHAIN_SPLITK) {
        c.args.lam = lam;
        c.args.L = K;
        c.args.S = 1;
        c.out = kOutLambda;
        if (use == LBI_ALGO_CHAIN_WAVE)
            return launch_chain_wave_bf16(c) == hipSuccess ? LBI_OK : LBI_ERR_HIP;
        if (use == LBI_ALGO_CHAIN_SPLITK) {
            c.hint = false;  // zero-padded tiles need no hint
            return launch_chain_ksplit_f32x(c) == hipSuccess ? LBI_OK : LBI_ERR_HIP;
        }
        return launch_chain_mode(c, dt, math) == hipSuccess ? LBI_OK : LBI_ERR_HIP;
    }

    // two-level scan: each segment folded (every composite kept, or its
    // aggregate only); the carries right to left; then every lambda_j at once
    // from the composites, or each segment scanned again from its carry
    char *w = (char *)ws;
    float *Pc = (float *)(w + p.offP);
    float *cc = b ? (float *)(w + p.offc) : nullptr;
    float *carry = (float *)(w + p.offcarry);
    c.args.L = p.L;
    c.args.S = p.S;
    c.args.Pout = Pc;
    c.args.cout = cc;
    c.args.agg_only = p.rescan ? 1 : 0;
    c.out = kOutComposite;
    // a segment's composites (and its lambda pass) have the width of the
    // segment's end, not lambda_K's: every column block
    c.ncol = r / 16;
    if (launch_chain_mode(c, dt, math) != hipSuccess)
        return LBI_ERR_HIP;
    if (launch_carry(Pc, cc, lamK, dt == LBI_BF16, carry, B, p.S, p.rescan ? p.S : K,
                     p.rescan ? 1 : p.L, r, c.stream) != hipSuccess)
        return LBI_ERR_HIP;
    if (!p.rescan)
        return launch_apply(Pc, cc, carry, lam, B, K, p.L, p.S, r, c.stream) == hipSuccess
                   ? LBI_OK
                   : LBI_ERR_HIP;
    c.args.Pout = nullptr;
    c.args.cout = nullptr;
    c.args.agg_only = 0;
    c.args.lam = lam;
    c.args.lamSeg = carry;
    c.out = kOutLambda;
    if (launch_chain_mode(c, dt, math) != hipSuccess)
        return LBI_ERR_HIP;
    return LBI_OK;
}

// ---- Phase 1 (synthetic region map) ----------------------------------------

constexpr int kRegionParts = 20;

struct RegionPlan {
    size_t off[kRegionParts];
    size_t bytes;
};

// Workspace parts, each 256-byte aligned: su, sa, d, cvec, xpart, xbar, sbar,
// gbar, p, sue, se, encv, zhat, isig, JencT (fp32) and P1, JdT, UT, dpT, TT (bf16).
RegionPlan region_plan(int64_t B, int64_t K, int64_t L, int32_t D, int32_t X, int32_t r)
{
    const size_t BK = (size_t)B * K, Br = (size_t)B * r, nch = (size_t)((L + 63) / 64);
    const size_t n[kRegionParts] = {
        BK * D * 4, BK * D * 4, BK * D * 4, BK * X * 4, (size_t)B * nch * D * 4,
        (size_t)B * D * 4, BK * X * 4, BK * X * 4, BK * D * 4, BK * D * 4, BK * D * 4,
        BK * r * 4, BK * r * 4, BK * 4, (size_t)K * Br * r * 4,
        (size_t)K * Br * D * 2, (size_t)K * Br * D * 2, (size_t)K * Br * X * 2,
        (size_t)K * Br * D * 2, (size_t)K * Br * D * 2};
    RegionPlan p;
    size_t o = 0;
    for (int i = 0; i < kRegionParts; ++i) {
        p.off[i] = o;
        o += align256(n[i]);
    }
    p.bytes = o;
    return p;
}

// The token-mixing block adds, for G (sequence, region) pairs at a time: s16,
// h16, Vt (bf16), s32, c32, g32, y32, wv, Tpart (fp32), S16 (bf16), after the
// parts above.
// G is what fits kSsmGroupBytes (at least 1, and few enough for a 1-D grid of
// either tangent product's 256 x 256 tiles); the second tangent product
// writes one partial sum per 256-row tile of a pair (nchunk of them).
constexpr int kSsmParts = 10;
constexpr size_t kSsmGroupBytes = (size_t)6 << 30;

struct SsmPlan {
    RegionPlan base;
    int64_t G;
    int32_t nchunk;
    size_t off[kSsmParts];
    size_t bytes;
};

SsmPlan ssm_plan(int64_t B, int64_t K, int64_t L, int32_t D, int32_t X, int32_t r)
{
    SsmPlan p;
    p.base = region_plan(B, K, L, D, X, r);
    const size_t LD = (size_t)L * D, LX = (size_t)L * X, Lr = (size_t)L * r;
    const size_t mtiles = (Lr + 255) / 256;  // the tangent products' row tiles
    const size_t pair = align256(LD * 2) + align256(LX * 2) + align256(Lr * X * 2) +
                        3 * align256(LD * 4) + align256(LX * 4) + align256((size_t)D * 4) +
                        align256(mtiles * r * D * 4) + align256(Lr * D * 2);
    int64_t G = (int64_t)(kSsmGroupBytes / pair);
    const int64_t BK = B * K;
    const size_t nct = (size_t)((X > D ? X : D) + 255) / 256;
    const int64_t tiles = (int64_t)(mtiles * nct);
    if (G > BK)
        G = BK;
    if (G > 65535)
        G = 65535;
    if (G > (((int64_t)1 << 31) - 1) / tiles)
        G = (((int64_t)1 << 31) - 1) / tiles;
    if (G < 1)
        G = 1;
    // (the second product writes one partial sum per row tile)
    const size_t nch = mtiles;
    p.G = G;
    p.nchunk = (int32_t)nch;
    const size_t g = (size_t)G;
    const size_t n[kSsmParts] = {g * LD * 2, g * LX * 2, g * Lr * X * 2, g * LD * 4,
                                 g * LD * 4, g * LX * 4, g * LD * 4, g * D * 4,
                                 g * nch * r * D * 4, g * Lr * D * 2};
    size_t o = p.base.bytes;
    for (int i = 0; i < kSsmParts; ++i) {
        p.off[i] = o;
        o += align256(n[i]);
    }
    p.bytes = o;
    return p;
}

bool region_sizes_ok(int64_t B, int64_t K, int64_t L, int32_t D, int32_t X, int32_t r)
{
    if (B < 0 || K < 1 || L < 1 || !supported_r(r))
        return false;
    if (D < 64 || D > 2048 || D % 64 != 0 || X < 128 || X > 8192 || X % 128 != 0)
        return false;
    // launch grids: the tangent products put B r / 128 row tiles in y and K in z
    if (B > 65535 || K > 65535 || L > ((int64_t)1 << 24) ||
        (B * r + 127) / 128 > 65535)
        return false;
    return B * K * (X / 128) < ((int64_t)1 << 31) - 1;
}

// the token-mixing block's first tangent product has L r rows: L r / 128 row
// tiles in a launch's y
bool ssm_sizes_ok(int64_t L, int32_t r) { return (L * r + 127) / 128 <= 65535; }

}  // namespace

namespace {
// Argument checks shared by both region blocks; ws_need is the workspace the
// block needs, decay its extra input (NULL for the token-wise block).
lbi_status region_check(const lbi_region_params *params, const float *decay, bool ssm,
                        const void *x_embed, const float *m, float *A, float *m_next, int64_t B,
                        int64_t K, int64_t L, int32_t D, int32_t r, void *workspace,
                        size_t workspace_bytes, size_t ws_need)
{
    if (!params)
        return LBI_ERR_NULL;
    if (B == 0)
        return LBI_OK;
    const lbi_region_params &p = *params;
    const void *ptrs[] = {p.W_d1, p.b_d1, p.W_d2, p.b_d2, p.W1, p.W2, p.W_e1, p.b_e1, p.W_e2,
                          p.b_e2, p.alpha, p.gamma, p.beta, x_embed, m, A};
    for (const void *q : ptrs)
        if (!q)
            return LBI_ERR_NULL;
    if (ssm && !decay)
        return LBI_ERR_NULL;
    for (const void *q : ptrs)
        if (misaligned(q))
            return LBI_ERR_ALIGN;
    if (misaligned(m_next) || misaligned(workspace) || misaligned(decay))
        return LBI_ERR_ALIGN;
    if (!workspace || workspace_bytes < ws_need)
        return LBI_ERR_WORKSPACE;
    const size_t nA = (size_t)B * K * r * r * 4, nm = (size_t)B * K * r * 4;
    const size_t nx = (size_t)B * L * D * 2;
    if (overlaps(A, nA, x_embed, nx) || overlaps(A, nA, m, nm) ||
        overlaps(A, nA, workspace, ws_need) || overlaps(m_next, nm, x_embed, nx) ||
        overlaps(m_next, nm, m, nm) || overlaps(m_next, nm, A, nA) ||
        overlaps(m_next, nm, workspace, ws_need) || overlaps(workspace, ws_need, m, nm) ||
        overlaps(workspace, ws_need, x_embed, nx))
        return LBI_ERR_ALIAS;
    if (ssm) {
        const size_t nd = (size_t)K * D * 4;
        if (overlaps(A, nA, decay, nd) || overlaps(m_next, nm, decay, nd) ||
            overlaps(workspace, ws_need, decay, nd))
            return LBI_ERR_ALIAS;
    }
    return LBI_OK;
}

// The launch arguments of both blocks (the token-wise block's workspace parts).
RegionArgs region_args(const lbi_region_params &p, const void *x_embed, const float *m, float *A,
                       float *m_next, int64_t B, int64_t K, int64_t L, int32_t D, int32_t X,
                       int32_t r, void *workspace, const RegionPlan &plan)
{
    RegionArgs q;
    memset(&q, 0, sizeof q);
    q.W_d1 = p.W_d1;
    q.W_d2 = p.W_d2;
    q.W1 = p.W1;
    q.W2 = p.W2;
    q.W_e1 = p.W_e1;
    q.W_e2 = p.W_e2;
    q.b_d1 = p.b_d1;
    q.b_d2 = p.b_d2;
    q.b_e1 = p.b_e1;
    q.b_e2 = p.b_e2;
    q.alpha = p.alpha;
    q.gamma = p.gamma;
    q.beta = p.beta;
    q.x_embed = x_embed;
    q.m = m;
    q.A = A;
    q.m_next = m_next;
    q.B = B;
    q.K = K;
    q.L = L;
    q.D = D;
    q.X = X;
    q.r = r;
    char *w = (char *)workspace;
    float **f32[15] = {&q.su,  &q.sa, &q.d,   &q.cvec, &q.xpart, &q.xbar, &q.sbar, &q.gbar,
                       &q.p,   &q.sue, &q.se, &q.encv, &q.zhat,  &q.isig, &q.JencT};
    for (int i = 0; i < 15; ++i)
        *f32[i] = (float *)(w + plan.off[i]);
    __bf16 **h16[5] = {&q.P1, &q.JdT, &q.UT, &q.dpT, &q.TT};
    for (int i = 0; i < 5; ++i)
        *h16[i] = (__bf16 *)(w + plan.off[15 + i]);
    return q;
}
}  // namespace

extern "C" {

size_t lbi_scan_backward_workspace_bytes_ex(int64_t B, int64_t K, int32_t r, lbi_dtype dt,
                                            lbi_algo algo)
{
    if (check_common(dt, LBI_MATH_DEFAULT, r, B, K) != LBI_OK || B == 0)
        return 0;
    if (!valid_algo(algo))
        return 0;
    const lbi_algo use = resolve_algo(algo, B, K, r, dt, LBI_MATH_DEFAULT);
    if (use == LBI_ALGO_TREE)
        // (sized for an affine term: enough with or without b)
        return r <= 64 && tree_possible(B, K, r) ? tree_plan(B, K, r, true).bytes : 0;
    if (use != LBI_ALGO_TWO_LEVEL || !two_level_possible(B, K))
        return 0;
    return two_level_plan(B, K, r).bytes;
}

size_t lbi_scan_backward_workspace_bytes(int64_t B, int64_t K, int32_t r, lbi_dtype dt)
{
    return lbi_scan_backward_workspace_bytes_ex(B, K, r, dt, LBI_ALGO_AUTO);
}

lbi_status lbi_scan_backward(const void *A, const void *b, const void *lambda_K, float *lambda,
                             int64_t B, int64_t K, int32_t r, lbi_dtype dt, void *workspace,
                             size_t workspace_bytes, lbi_stream_t stream)
{
    return scan_impl(A, b, lambda_K, lambda, B, K, r, dt, workspace, workspace_bytes, stream,
                     nullptr, LBI_MATH_DEFAULT, LBI_ALGO_AUTO);
}

lbi_status lbi_scan_backward_widths(const void *A, const void *b, const void *lambda_K,
                                    float *lambda, int64_t B, int64_t K, int32_t r, lbi_dtype dt,
                                    void *workspace, size_t workspace_bytes, lbi_stream_t stream,
                                    const int32_t *widths_host)
{
    return scan_impl(A, b, lambda_K, lambda, B, K, r, dt, workspace, workspace_bytes, stream,
                     widths_host, LBI_MATH_DEFAULT, LBI_ALGO_AUTO);
}

lbi_status lbi_scan_backward_ex(const void *A, const void *b, const void *lambda_K,
                                float *lambda, int64_t B, int64_t K, int32_t r, lbi_dtype dt,
                                void *workspace, size_t workspace_bytes, lbi_stream_t stream,
                                const int32_t *widths_host, lbi_math math, lbi_algo algo)
{
    return scan_impl(A, b, lambda_K, lambda, B, K, r, dt, workspace, workspace_bytes, stream,
                     widths_host, math, algo);
}

lbi_status lbi_scan_suffix_products(const void *A, const void *b, float *P, float *c, int64_t B,
                                    int64_t K, int32_t r, lbi_dtype dt, lbi_stream_t stream,
                                    const int32_t *widths_host, lbi_math math)
{
    lbi_status st = check_common(dt, math, r, B, K);
    if (st != LBI_OK)
        return st;
    if (B == 0)
        return LBI_OK;
    if (!A || !P)
        return LBI_ERR_NULL;
    if (misaligned(A) || misaligned(b) || misaligned(P) || misaligned(c))
        return LBI_ERR_ALIGN;
    const size_t esz = dt == LBI_F32 ? 4 : 2;
    const size_t nA = (size_t)B * K * r * r * esz, nb = b ? (size_t)B * K * r * esz : 0;
    const size_t nP = (size_t)B * K * r * r * sizeof(float);
    const size_t nc = c ? (size_t)B * K * r * sizeof(float) : 0;
    if (overlaps(P, nP, A, nA) || overlaps(P, nP, b, nb) || overlaps(c, nc, A, nA) ||
        overlaps(c, nc, b, nb) || overlaps(c, nc, P, nP))
        return LBI_ERR_ALIAS;
    ChainLaunch cl;
    memset(&cl, 0, sizeof cl);
    cl.args.A = A;
    cl.args.b = b;
    cl.args.Pout = P;
    cl.args.cout = c;
    cl.args.K = K;
    cl.args.L = K;
    cl.args.S = 1;
    cl.B = B;
    cl.r = r;
    cl.aff = b != nullptr;
    cl.out = kOutComposite;
    cl.stream = (hipStream_t)stream;
    if (!encode_widths(widths_host, K, r, cl))
        return LBI_ERR_SHAPE;
    cl.ncol = r / 16;
    return launch_chain_mode(cl, dt, math) == hipSuccess ? LBI_OK : LBI_ERR_HIP;
}

lbi_status lbi_scan_backward_ragged(const void *A, const void *b, const void *lambda_K,
                                    float *lambda, int64_t B, int64_t K,
                                    const int32_t *widths_host, lbi_dtype dt, lbi_stream_t stream,
                                    lbi_math math)
{
    if (dt != LBI_F32 && dt != LBI_BF16)
        return LBI_ERR_DTYPE;
    if (B < 0 || K < 1 || K > LBI_MAX_HINT_K)
        return LBI_ERR_SHAPE;
    if (!widths_host)
        return LBI_ERR_NULL;
    int32_t rmax = 0;
    for (int64_t k = 0; k <= K; ++k) {
        const int32_t wk = widths_host[k];
        if (wk < 16 || wk > 128 || wk % 16 != 0)
            return LBI_ERR_SHAPE;
        rmax = wk > rmax ? wk : rmax;
    }
    const int32_t R = rmax <= 16 ? 16 : (rmax <= 32 ? 32 : (rmax <= 64 ? 64 : 128));
    lbi_status st = check_common(dt, math, R, B, K);
    if (st != LBI_OK)
        return st;
    int64_t totA = 0, totR = 0;
    for (int64_t j = 0; j < K; ++j) {
        totA += (int64_t)widths_host[j] * widths_host[j + 1];
        totR += widths_host[j];
    }
    if (B == 0)
        return LBI_OK;
    if (!A || !lambda_K || !lambda)
        return LBI_ERR_NULL;
    if (misaligned(A) || misaligned(b) || misaligned(lambda_K) || misaligned(lambda))
        return LBI_ERR_ALIGN;
    const size_t esz = dt == LBI_F32 ? 4 : 2;
    const size_t nA = (size_t)B * totA * esz, nb = b ? (size_t)B * totR * esz : 0;
    const size_t nl = (size_t)B * widths_host[K] * esz, nout = (size_t)B * totR * sizeof(float);
    if (overlaps(lambda, nout, A, nA) || overlaps(lambda, nout, b, nb) ||
        overlaps(lambda, nout, lambda_K, nl))
        return LBI_ERR_ALIAS;
    ChainLaunch c;
    memset(&c, 0, sizeof c);
    c.args.A = A;
    c.args.b = b;
    c.args.lamK = lambda_K;
    c.args.lam = lambda;
    c.args.K = K;
    c.args.L = K;
    c.args.S = 1;
    c.args.compact = 1;
    c.args.totalA = (int32_t)totA;
    c.args.totalR = (int32_t)totR;
    c.B = B;
    c.r = R;
    c.aff = b != nullptr;
    c.out = kOutLambda;
    c.stream = (hipStream_t)stream;
    if (!encode_widths(widths_host, K, R, c) || !c.hint)
        return LBI_ERR_SHAPE;
    // bf16 in the default arithmetic, widths the LDS-ring kernel takes: that
    // kernel (it reads the compact tiles block by block)
    if (dt == LBI_BF16 && math != LBI_MATH_BF16_SINGLE) {
        const RingPlan rp = ring_plan(widths_host, K, R);
        if (rp.ok) {
            c.args.ring = rp.ring;
            c.args.pitch = R;
            return launch_chain_ring_bf16(c, rp.maxb) == hipSuccess ? LBI_OK : LBI_ERR_HIP;
        }
    }
    return launch_chain_mode(c, dt, math) == hipSuccess ? LBI_OK : LBI_ERR_HIP;
}

size_t lbi_region_jacobians_workspace_bytes(int64_t B, int64_t K, int64_t L, int32_t D,
                                            int32_t X, int32_t r)
{
    if (!region_sizes_ok(B, K, L, D, X, r))
        return 0;
    return region_plan(B, K, L, D, X, r).bytes;
}


lbi_status lbi_region_jacobians(const lbi_region_params *params, const void *x_embed,
                                const float *m, float *A, float *m_next, int64_t B, int64_t K,
                                int64_t L, int32_t D, int32_t X, int32_t r, void *workspace,
                                size_t workspace_bytes, lbi_stream_t stream)
{
    if (!region_sizes_ok(B, K, L, D, X, r))
        return r > 0 && !supported_r(r) ? LBI_ERR_UNSUPPORTED_R : LBI_ERR_SHAPE;
    const RegionPlan plan = region_plan(B, K, L, D, X, r);
    const lbi_status st = region_check(params, nullptr, false, x_embed, m, A, m_next, B, K, L, D,
                                       r, workspace, workspace_bytes, plan.bytes);
    if (st != LBI_OK || B == 0)
        return st;
    const RegionArgs q = region_args(*params, x_embed, m, A, m_next, B, K, L, D, X, r, workspace,
                                     plan);
    return launch_region_jacobians(q, (hipStream_t)stream) == hipSuccess ? LBI_OK : LBI_ERR_HIP;
}

size_t lbi_region_jacobians_ssm_workspace_bytes(int64_t B, int64_t K, int64_t L, int32_t D,
                                                int32_t X, int32_t r)
{
    if (!region_sizes_ok(B, K, L, D, X, r) || !ssm_sizes_ok(L, r))
        return 0;
    return ssm_plan(B, K, L, D, X, r).bytes;
}

lbi_status lbi_region_jacobians_ssm(const lbi_region_params *params, const float *decay,
                                    const void *x_embed, const float *m, float *A, float *m_next,
                                    int64_t B, int64_t K, int64_t L, int32_t D, int32_t X,
                                    int32_t r, void *workspace, size_t workspace_bytes,
                                    lbi_stream_t stream)
{
    if (!region_sizes_ok(B, K, L, D, X, r) || !ssm_sizes_ok(L, r))
        return r > 0 && !supported_r(r) ? LBI_ERR_UNSUPPORTED_R : LBI_ERR_SHAPE;
    const SsmPlan plan = ssm_plan(B, K, L, D, X, r);
    const lbi_status st = region_check(params, decay, true, x_embed, m, A, m_next, B, K, L, D, r,
                                       workspace, workspace_bytes, plan.bytes);
    if (st != LBI_OK || B == 0)
        return st;
    RegionArgs q = region_args(*params, x_embed, m, A, m_next, B, K, L, D, X, r, workspace,
                               plan.base);
    char *w = (char *)workspace;
    q.decay = decay;
    q.G = plan.G;
    q.nchunk = plan.nchunk;
    q.s16 = (__bf16 *)(w + plan.off[0]);
    q.h16 = (__bf16 *)(w + plan.off[1]);
    q.Vt = (__bf16 *)(w + plan.off[2]);
    q.s32 = (float *)(w + plan.off[3]);
    q.c32 = (float *)(w + plan.off[4]);
    q.g32 = (float *)(w + plan.off[5]);
    q.y32 = (float *)(w + plan.off[6]);
    q.wv = (float *)(w + plan.off[7]);
    q.Tpart = (float *)(w + plan.off[8]);
    q.S16 = (__bf16 *)(w + plan.off[9]);
    return launch_region_jacobians_ssm(q, (hipStream_t)stream) == hipSuccess ? LBI_OK
                                                                             : LBI_ERR_HIP;
}

lbi_status lbi_matrix_norms(const void *M, int64_t n, int32_t r, lbi_dtype dt, float *spec,
                            float *fro, lbi_stream_t stream)
{
    // the shape checks of a scan over n chains of one slot
    lbi_status st = check_common(dt, LBI_MATH_DEFAULT, r, n, 1);
    if (st != LBI_OK)
        return st;
    if (n == 0)
        return LBI_OK;
    if (!M || (!spec && !fro))
        return LBI_ERR_NULL;
    if (misaligned(M) || misaligned(spec) || misaligned(fro))
        return LBI_ERR_ALIGN;
    const size_t esz = dt == LBI_F32 ? 4 : 2;
    const size_t nM = (size_t)n * r * r * esz, nout = (size_t)n * sizeof(float);
    if (overlaps(spec, nout, M, nM) || overlaps(fro, nout, M, nM) ||
        overlaps(spec, nout, fro, nout))
        return LBI_ERR_ALIAS;
    return launch_norms(M, dt == LBI_BF16, n, r, spec, fro, (hipStream_t)stream) == hipSuccess
               ? LBI_OK
               : LBI_ERR_HIP;
}

lbi_status lbi_scan_backward_streaming(const void *A, const void *b, const void *lambda_K,
                                       float *lambda, int64_t B, int64_t K, int32_t r,
                                       lbi_dtype dt, lbi_stream_t stream,
                                       const int32_t *widths_host, lbi_math math,
                                       uint32_t *progress, int32_t chunk,
                                       uint64_t *publish_clock)
{
    lbi_status st = check_common(dt, math, r, B, K);
    if (st != LBI_OK)
        return st;
    if (chunk < 1 || K > (int64_t)UINT32_MAX)  // the counts are 32-bit
        return LBI_ERR_SHAPE;
    if (B == 0)
        return LBI_OK;
    if (!A || !lambda_K || !lambda || !progress)
        return LBI_ERR_NULL;
    if (misaligned(A) || misaligned(b) || misaligned(lambda_K) || misaligned(lambda) ||
        ((uintptr_t)progress & 3u) || ((uintptr_t)publish_clock & 7u))
        return LBI_ERR_ALIGN;
    const size_t esz = dt == LBI_F32 ? 4 : 2;
    const size_t nA = (size_t)B * K * r * r * esz, nb = b ? (size_t)B * K * r * esz : 0;
    const size_t nl = (size_t)B * r * esz, nout = (size_t)B * K * r * sizeof(float);
    const size_t np = (size_t)B * sizeof(uint32_t);
    const int64_t npub = (K + chunk - 1) / chunk;
    const size_t nc = publish_clock ? (size_t)B * npub * sizeof(uint64_t) : 0;
    if (overlaps(lambda, nout, A, nA) || overlaps(lambda, nout, b, nb) ||
        overlaps(lambda, nout, lambda_K, nl) || overlaps(progress, np, A, nA) ||
        overlaps(progress, np, b, nb) || overlaps(progress, np, lambda_K, nl) ||
        overlaps(progress, np, lambda, nout) || overlaps(publish_clock, nc, A, nA) ||
        overlaps(publish_clock, nc, b, nb) || overlaps(publish_clock, nc, lambda_K, nl) ||
        overlaps(publish_clock, nc, lambda, nout) || overlaps(publish_clock, nc, progress, np))
        return LBI_ERR_ALIAS;
    ChainLaunch c;
    memset(&c, 0, sizeof c);
    c.args.A = A;
    c.args.b = b;
    c.args.lamK = lambda_K;
    c.args.lam = lambda;
    c.args.K = K;
    c.args.L = K;
    c.args.S = 1;
    c.args.progress = progress;
    c.args.pchunk = chunk;
    c.args.npub = npub;
    c.args.pub_clock = publish_clock;
    c.B = B;
    c.r = r;
    c.aff = b != nullptr;
    c.out = kOutLambda;
    c.stream = (hipStream_t)stream;
    if (!encode_widths(widths_host, K, r, c))
        return LBI_ERR_SHAPE;
    return launch_chain_mode(c, dt, math) == hipSuccess ? LBI_OK : LBI_ERR_HIP;
}

lbi_status lbi_wait_progress(const uint32_t *progress, int64_t B, uint32_t target,
                             int64_t max_polls, uint32_t *released, uint64_t *release_clock,
                             lbi_stream_t stream)
{
    if (B < 0 || max_polls < 1)
        return LBI_ERR_SHAPE;
    if (B > 0 && !progress)
        return LBI_ERR_NULL;
    if (((uintptr_t)progress & 3u) || ((uintptr_t)released & 3u) ||
        ((uintptr_t)release_clock & 7u))
        return LBI_ERR_ALIGN;
    const size_t np = (size_t)B * sizeof(uint32_t);
    if (overlaps(released, 4, progress, np) || overlaps(release_clock, 8, progress, np) ||
        overlaps(released, 4, release_clock, 8))
        return LBI_ERR_ALIAS;
    return launch_wait_progress(progress, B, target, max_polls, released, release_clock,
                                (hipStream_t)stream) == hipSuccess
               ? LBI_OK
               : LBI_ERR_HIP;
}

lbi_status lbi_scan_backward_noalloc(const void *A, const void *b, const void *lambda_K,
                                     float *lambda, int64_t B, int64_t K, int32_t r,
                                     lbi_dtype dt, lbi_stream_t stream,
                                     const int32_t *widths_host, lbi_math math, lbi_algo algo)
{
    return scan_impl(A, b, lambda_K, lambda, B, K, r, dt, nullptr, 0, stream, widths_host, math,
                     algo, true);
}

const char *lbi_status_string(lbi_status s)
{
    switch (s) {
    case LBI_OK: return "LBI_OK";
    case LBI_ERR_NULL: return "LBI_ERR_NULL: a required pointer is NULL";
    case LBI_ERR_SHAPE: return "LBI_ERR_SHAPE: bad B, K, size or widths";
    case LBI_ERR_DTYPE: return "LBI_ERR_DTYPE: unknown dtype, math mode or algorithm";
    case LBI_ERR_UNSUPPORTED_R: return "LBI_ERR_UNSUPPORTED_R: r must be 16, 32, 64 or 128";
    case LBI_ERR_WORKSPACE: return "LBI_ERR_WORKSPACE: workspace missing or too small";
    case LBI_ERR_HIP: return "LBI_ERR_HIP: the HIP runtime refused the launch";
    case LBI_ERR_ALIGN: return "LBI_ERR_ALIGN: a pointer is not 16-byte aligned";
    case LBI_ERR_ALIAS: return "LBI_ERR_ALIAS: an output overlaps an input";
    case LBI_ERR_SCRATCH:
        return "LBI_ERR_SCRATCH: the call needs more than the library's static scratch array "
               "(LBI_NOALLOC_SCRATCH_BYTES)";
    }
    return "unknown lbi_status";
}

int lbi_abi_version(void) { return LBI_ABI_VERSION; }

}  // extern "C"
