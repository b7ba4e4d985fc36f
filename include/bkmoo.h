/*
 * bkmoo — bucket-level gradient-conflict resolution on MI355X (gfx950).
 *
 * The operation (Section 3.2 and Algorithm 1 of "Multilingual Fine-Tuning
 * via Localized Gradient Conflict Resolution"): the flattened parameter
 * vector is cut into B contiguous buckets; every language (task) i of K has
 * its own gradient x_i over all N parameters.  For each bucket b the local
 * gradient set is the K slices x_i[o_b : o_{b+1}], a small multi-objective
 * problem is solved on that set alone, and the bucket's update is a weighted
 * sum of the slices,
 *
 *     d[o_b : o_{b+1}] = sum_i w_{b,i} x_i[o_b : o_{b+1}],
 *
 * with the updates of all buckets concatenated into d (Algorithm 1, final
 * step).  Every bucket-level method only sees its gradients through their
 * inner products, so the work splits into
 *
 *     gram    G_b[i][j] = <x_i, x_j> over the bucket      (streams K*N)
 *     solve   G_b -> w_b (MGDA, PCGrad, CAGrad, or mean)  (K x K work)
 *     combine d = sum_i w_{b,i} x_i                        (streams K*N, writes N)
 *
 * and resolve runs the three in order on one stream.
 *
 * Notation: the paper writes T for the number of languages and K for the
 * number of buckets; this interface writes K for the languages and B for the
 * buckets.
 *
 * Conventions shared by every entry point
 *   - Pointers are DEVICE pointers unless marked (host).  The caller owns and
 *     allocates every buffer; the library never allocates, frees or
 *     synchronises inside these calls, and all work is queued on `stream`
 *     (asynchronous; results are valid once the stream reaches that point).
 *   - Device pointers must be memory of the current HIP device (hipGetDevice)
 *     and `stream` must belong to it: launch grids are sized from that
 *     device's compute units and occupancy.  The library cannot tell a host
 *     or foreign pointer from a device one; passing one is undefined (a GPU
 *     memory fault).
 *   - grads is a HOST array of K device pointers, one per task, each to N
 *     elements of dtype `dt`.  A contiguous [K][N] buffer is passed as
 *     base + i*N*elem_size.  Rows need natural alignment (4 bytes for f32,
 *     2 for bf16); 16-byte alignment of every row at the same phase enables
 *     128-bit loads, otherwise a scalar path is used.
 *   - bucket_offsets is int64[B+1] in device memory with o_0 = 0, o_B = N and
 *     o_b <= o_{b+1} (empty buckets are allowed).  Offsets are checked on the
 *     device; invalid offsets set BKMOO_DEVERR_OFFSETS in the workspace error
 *     word (see bkmoo_read_device_error), make every Gram entry NaN and leave
 *     `out` untouched.  No memory outside [0, N) is ever touched.
 *   - Inputs are converted exactly to fp32; inner products accumulate in fp32
 *     per lane and in fp64 across lanes, waves and chunks, in a fixed order:
 *     results are bitwise reproducible for identical inputs on the same
 *     device model, independent of the launch grid.
 *   - Non-finite inputs propagate (a NaN in a bucket makes its Gram, weights
 *     and update NaN); nothing is filtered.
 *   - Synchronous argument errors are returned before anything is queued.
 *     HIP launch failures return BKMOO_EHIP.
 *   - Calls are re-entrant; concurrent calls must not share a workspace.
 */
#ifndef BKMOO_H
#define BKMOO_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  BKMOO_OK = 0,
  BKMOO_EINVAL = -1,        /* bad argument: null pointer, size, enum or hyper-parameter */
  BKMOO_EUNSUPPORTED = -2,  /* well-formed but unsupported (e.g. K outside [2, 16]) */
  BKMOO_EWORKSPACE = -3,    /* ws_bytes smaller than bkmoo_workspace_size() */
  BKMOO_EHIP = -4           /* a HIP call or kernel launch failed */
} bkmoo_status;

typedef enum { BKMOO_F32 = 0, BKMOO_BF16 = 1 } bkmoo_dtype;

/* Bucket-level strategy M of Algorithm 1, plus the plain average. */
typedef enum {
  BKMOO_MGDA = 0,    /* min-norm point of the bucket's gradient hull, Eq. (shard-mgda) */
  BKMOO_PCGRAD = 1,  /* projection of conflicting pairs, Eq. (pcgrad_proj), Algorithm 1 */
  BKMOO_CAGRAD = 2,  /* conflict-averse direction in a ball around the mean, Eq. (cagrad) */
  BKMOO_MEAN = 3,    /* averaged gradient (1/K) sum_i x_i, Section 2.1 */
  BKMOO_MGDA_EXACT = 4,   /* MGDA's min-norm point solved exactly (K <= 10) */
  BKMOO_CAGRAD_EXACT = 5  /* CAGrad's dual solved exactly (K <= 10) */
} bkmoo_method;

/* Device error word bits (bkmoo_read_device_error). */
#define BKMOO_DEVERR_OFFSETS 0x1u /* bucket offsets rejected */
#define BKMOO_DEVERR_TIMEOUT 0x2u /* a bounded wait of the hybrid path expired: the update is invalid
                                     (buckets whose wait expired get NaN weights and a NaN update) */

/* Layout of T sets of per-slice partial Gram matrices (bkmoo_gram_reduce). */
typedef enum {
  BKMOO_SLICES_RANK_MAJOR = 0,   /* partial[t][b][K][K]: T gathered per-rank sets */
  BKMOO_SLICES_BUCKET_MAJOR = 1  /* partial[b][t][K][K]: bkmoo_gram over slice offsets */
} bkmoo_slice_layout;

/* How bkmoo_resolve runs the step (bkmoo_resolve_path).  Other values are
 * rejected. */
typedef enum {
  BKMOO_PATH_TWO_PASS = 1, /* Gram pass, solve, combine pass: reads the gradients twice */
  BKMOO_PATH_HYBRID = 3,   /* one cooperative kernel, part of each bucket held on chip, the next
                              bucket's Gram overlapping this one's solve */
  BKMOO_PATH_REFILL = 4    /* one cooperative kernel (K <= 10), part of each bucket held on chip in
                              one buffer refilled with the next bucket as it is combined */
} bkmoo_path;

/* Hyper-parameters of the solve step (host struct). */
typedef struct {
  /* Frank-Wolfe iterations for MGDA and CAGrad (fixed count, no early
   * exit), >= 0.  The usual value is 20. */
  int32_t max_iter;
  /* CAGrad conflict-aversion c in [0, 1): the update stays within
   * c * ||mean gradient|| of the mean gradient (Eq. cagrad); Appendix E
   * uses 0.5. */
  double cagrad_c;
  /* PCGrad visiting order, device int8 [B][K][K-1]: row (b, t) lists the
   * other tasks j != t in the order task t is projected against them (the
   * "random order" of Algorithm 1, drawn by the caller).  NULL visits them
   * in ascending order.  A row that is not a permutation of {j != t} makes
   * that bucket's weights NaN. */
  const int8_t *pcgrad_order;
} bkmoo_hparams;

/*
 * bkmoo_workspace_size — bytes of device workspace that bkmoo_gram,
 * bkmoo_combine and bkmoo_resolve need for (K, N, B, dt).  The size is an
 * upper bound that depends on these four values only (about 8 bytes per
 * bucket plus 8*K*(K+1)/2 bytes per chunk of a few thousand elements).
 * Workspace contents need no initialisation and are scratch between calls,
 * except the error word, which the next call clears.
 * Returns BKMOO_EINVAL for K < 2, N < 0, B < 1, bad dt or a null `bytes`
 * (host), BKMOO_EUNSUPPORTED for K > 16.
 */
bkmoo_status bkmoo_workspace_size(int32_t K, int64_t N, int32_t B, bkmoo_dtype dt, size_t *bytes);

/*
 * bkmoo_gram — per-bucket Gram matrices (the inner products every
 * bucket-level method is defined through: ||sum_t a_t g_t||^2 = a^T G a in
 * Eq. (shard-mgda); <g_i, g_j> in PCGrad's conflict test, Section 3.2).
 *
 *   gram (out) fp64 [B][K][K], row-major, symmetric:
 *        gram[b][i][j] = sum_{n in [o_b, o_{b+1})} x_i[n] * x_j[n].
 * Each input row is read once with 128-bit loads.
 */
bkmoo_status bkmoo_gram(int32_t K, const void *const *grads, bkmoo_dtype dt, int64_t N, int32_t B,
                        const int64_t *bucket_offsets, double *gram, void *workspace,
                        size_t ws_bytes, hipStream_t stream);

/*
 * bkmoo_solve — the small per-bucket MOO problem, one wavefront per bucket,
 * in fp64, from the Gram matrices alone.
 *
 *   gram    (in)  fp64 [B][K][K] (as written by bkmoo_gram)
 *   weights (out) fp32 [B][K]: the combine coefficients, d_b = sum_i w_{b,i} g_{b,i}
 *   aux     (out, may be NULL) fp64 [B][K]: the method's own variable
 *
 *   MGDA   (Eq. shard-mgda over the simplex): Frank-Wolfe started on the best
 *          pair of tasks, argmin vertex with lowest-index ties, exact line
 *          search, hp->max_iter iterations.  weights = aux = alpha.  For K=2
 *          the start is already the exact minimiser.
 *   PCGrad (Algorithm 1): d_t = g_t, projected off each g_j (visiting
 *          order from hp->pcgrad_order) whenever <d_t, g_j> < 0; d = sum_t d_t,
 *          tracked exactly as coefficients on the original g_i.
 *          weights = aux = those coefficients (a sum, not a mean).
 *   CAGrad (Eq. cagrad per bucket): the dual min over the simplex of
 *          <g_w, g_avg> + c||g_avg|| ||g_w||, Frank-Wolfe from the uniform
 *          point with exact line search, hp->max_iter iterations; then
 *          d = g_avg + c||g_avg|| g_w/||g_w||, i.e. weights = 1/K + r w/||g_w||
 *          (1/K when r = 0 or g_w vanishes); aux = w.
 *   MEAN   weights = aux = 1/K.
 *   MGDA_EXACT / CAGRAD_EXACT  the same two problems solved exactly, K <= 10,
 *          by enumerating the 2^K - 1 supports S (one wavefront per bucket,
 *          one support per lane at a time, Gaussian elimination with partial
 *          pivoting per support; a support with an exactly zero pivot is
 *          skipped).  Supports are ranked by size, then lexicographically.
 *          MGDA: on S, G_SS a = mu 1 with 1^T a = 1 (G divided by its largest
 *          diagonal entry); kept if a >= -1e-10, |1^T a - 1| <= 1e-9 and,
 *          clipped and renormalised, (G a)_t >= a^T G a - 1e-9 for every t;
 *          the first kept support in rank order wins unless a later one is
 *          lower by more than 1e-12; none kept -> 5000 Frank-Wolfe
 *          iterations.  weights = aux = alpha.  CAGrad: the vertices and, for
 *          r > 0 and |S| >= 2, both roots of the stationarity conditions on
 *          S (v_S = G_SS^-1 (lam 1 - b_S) / r with v^T G v = 1), kept if
 *          v >= -1e-12 and 1^T v > 0, normalised onto the simplex; least dual
 *          value wins, first in rank order on ties (vertices, then supports,
 *          smaller root first); weights and aux as for CAGRAD.  max_iter is
 *          ignored; CAGRAD_EXACT needs hp->cagrad_c.
 * `hp` (host) may be NULL for MEAN and MGDA_EXACT; PCGrad ignores max_iter
 * and c.  BKMOO_EUNSUPPORTED for an exact method with K > 10.
 */
bkmoo_status bkmoo_solve(int32_t K, int32_t B, const double *gram, bkmoo_method method,
                         const bkmoo_hparams *hp, float *weights, double *aux, hipStream_t stream);

/*
 * bkmoo_combine — the resolved update of every bucket, concatenated
 * (Algorithm 1: d_(k) per strategy, then d = [d_(1), ..., d_(K)]).
 *
 *   weights (in)  fp32 [B][K]
 *   out     (out) N elements of out_dt, out[n] = sum_i w_{b,i} x_i[n] for n in
 *           bucket b, summed in task order: an fp32 FMA chain for an fp32
 *           output; for a bf16 output an fp64 chain (exact products) rounded
 *           once to nearest-even bf16 (via round-to-odd fp32).
 * `out` may be exactly one of the grads rows (in-place update); any other
 * overlap with the inputs is undefined.
 */
bkmoo_status bkmoo_combine(int32_t K, const void *const *grads, bkmoo_dtype dt, int64_t N, int32_t B,
                           const int64_t *bucket_offsets, const float *weights, void *out,
                           bkmoo_dtype out_dt, void *workspace, size_t ws_bytes, hipStream_t stream);

/*
 * bkmoo_resolve — gram, solve and combine in order on `stream` (one pass of
 * Algorithm 1's per-bucket loop over all buckets), with no host
 * synchronisation.  gram, weights and aux may be NULL, in which case the
 * intermediate values live in the workspace only.
 *
 * Two implementations, same definitions and tolerances:
 *   two-pass  the kernels of bkmoo_gram, bkmoo_solve and bkmoo_combine;
 *             results equal those three calls bitwise.
 *   hybrid    (K <= 8, 16-byte-phase-aligned rows and output) one
 *             cooperative kernel in which the Gram pass of bucket b+1 runs
 *             while bucket b is solved; part of each bucket (about half at
 *             K <= 4, less for more tasks) stays on chip between its Gram
 *             and its combine and the rest is read again (partly from the
 *             last-level cache).  The Gram sums run in a different (also
 *             fixed) order, so results agree with the two-pass path to
 *             rounding, not bitwise; they depend on the device's CU count
 *             and, for K >= 4 with MGDA or CAGrad, on the segment layout
 *             the method selects (deterministic for given arguments).
 *             Its cross-workgroup hand-off waits are bounded: if one
 *             expires the call still completes, sets BKMOO_DEVERR_TIMEOUT in
 *             the workspace error word, and the buckets concerned get NaN
 *             weights and a NaN update.
 *   refill    (K <= 10, aligned as for hybrid) one cooperative kernel that
 *             keeps up to twice the hybrid's share of each bucket on chip
 *             in a single buffer: the part of bucket b+1 it does not keep
 *             is read while bucket b is solved, then each kept vector of
 *             bucket b is combined and replaced by bucket b+1's.  Its data
 *             workgroups form G groups (G = clamp(round(180 MiB / bucket
 *             size, all rows), 1, 32), at most B) and group g takes buckets
 *             g, g+G, ..., so small buckets hide their hand-off too.
 *             Rounding, determinism and bounded waits as for hybrid (its
 *             segments also depend on G).
 * Automatic choice, with L the estimated solve latency (0.07 K us per MGDA
 * iteration, 0.22 K us per CAGrad iteration, 0.1 K^2 us for PCGrad, 0 for
 * the mean): hybrid (K <= 8) is eligible for at least 8 buckets of which at
 * least 10% stays on chip, averaging (all K rows) at least max(24, 6 K) MiB
 * plus 4 MiB per us of L; refill (K <= 10) for at least 8 buckets whose
 * round of G buckets holds at least 64 + 2 L MiB and, for G > 1, at most
 * 300 MiB (a round the Infinity Cache still serves).  Hybrid where it
 * is eligible, except refill for K = 3 and for K <= 4 with L >= 4 us; else
 * refill where eligible; else the two passes.  Exact solvers never take a cooperative
 * path.
 * bkmoo_resolve_path reports the choice; bkmoo_set_resolve_path forces one.
 */
bkmoo_status bkmoo_resolve(int32_t K, const void *const *grads, bkmoo_dtype dt, int64_t N, int32_t B,
                           const int64_t *bucket_offsets, bkmoo_method method,
                           const bkmoo_hparams *hp, void *out, bkmoo_dtype out_dt, double *gram,
                           float *weights, double *aux, void *workspace, size_t ws_bytes,
                           hipStream_t stream);

/*
 * bkmoo_resolve_noalloc — bkmoo_resolve for callers that cannot allocate
 * device memory or hand the library a workspace (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation).  Same
 * arguments as bkmoo_resolve minus workspace/ws_bytes, same paths, results
 * and errors; the workspace is a fixed array of the library instead:
 *   - 96 MiB per device (file-scope device memory of the library, present
 *     on every device the library runs on until the process ends).  A call
 *     whose bkmoo_workspace_size(K, N, B, dt) exceeds it returns
 *     BKMOO_EWORKSPACE before anything is queued.  The size is about
 *     K(K+1)/2 * 8 bytes per chunk of 16-32K elements: 19 MiB for K=4 bf16
 *     over 8.03B parameters in 25 MiB buckets, 68 MiB for K=8 at that
 *     shape, 57 MiB for K=10 fp32 over 1.72B parameters in 1 MiB buckets.
 *   - No allocation, free or synchronisation: the first call on a device
 *     looks up that device's address of the array (hipGetSymbolAddress)
 *     with that device current; every call is then launches on `stream`.
 *   - Every call on a device shares that device's array, which keeps the
 *     last call's contents (each call clears what must start at zero):
 *     calls that overlap in time on one device race and give undefined
 *     results.  Serialise them (one stream, or events).
 *   - The device error word lives in the array and cannot be read back;
 *     invalid offsets still make the Gram matrices NaN and a timeout of the
 *     hybrid path still makes the affected weights and update NaN.
 */
bkmoo_status bkmoo_resolve_noalloc(int32_t K, const void *const *grads, bkmoo_dtype dt, int64_t N,
                                   int32_t B, const int64_t *bucket_offsets, bkmoo_method method,
                                   const bkmoo_hparams *hp, void *out, bkmoo_dtype out_dt, double *gram,
                                   float *weights, double *aux, hipStream_t stream);

/*
 * bkmoo_slice_offsets — cut every bucket into T contiguous slices: slice t
 * of bucket b is [o_b + floor(t n_b / T), o_b + floor((t+1) n_b / T)),
 * n_b = o_{b+1} - o_b, the piece rank t of T would hold after the ranks
 * exchange bucket slices.  Inner products add over disjoint pieces
 * (Eq. decomp), so a bucket's Gram matrix is the sum of its slices'.
 *
 *   bucket_offsets (in)  device int64 [B+1]
 *   slice_offsets  (out) device int64 [B*T+1], bucket-major: bucket b's
 *                  slices 0..T-1 are entries b*T .. b*T+T; usable as the
 *                  bucket offsets of bkmoo_gram with B*T buckets
 *
 * Asynchronous on `stream`; the offsets are not validated here (bkmoo_gram
 * validates what it is given).  BKMOO_EINVAL for B < 1, T < 1, B*T beyond
 * int32 or a null pointer.
 */
bkmoo_status bkmoo_slice_offsets(int32_t B, int32_t T, const int64_t *bucket_offsets,
                                 int64_t *slice_offsets, hipStream_t stream);

/*
 * bkmoo_gram_reduce — add T sets of per-slice partial Gram matrices in
 * slice (rank) order t = 0, 1, ..., T-1, the same order on every rank, so
 * every rank gets the same Gram matrices bit for bit:
 *   gram[b] = partial(0, b) + partial(1, b) + ... + partial(T-1, b)
 *
 *   partial (in)  device fp64, `layout`: BKMOO_SLICES_RANK_MAJOR
 *                 [T][B][K][K] (the gathered per-rank sets) or
 *                 BKMOO_SLICES_BUCKET_MAJOR [B][T][K][K] (bkmoo_gram over
 *                 bkmoo_slice_offsets)
 *   gram    (out) device fp64 [B][K][K]; must not overlap `partial`
 *
 * Asynchronous on `stream`.  BKMOO_EINVAL for K < 2, B < 1, T < 1, a null
 * pointer or an unknown layout; BKMOO_EUNSUPPORTED for K > 16.
 */
bkmoo_status bkmoo_gram_reduce(int32_t K, int32_t B, int32_t T, const double *partial,
                               bkmoo_slice_layout layout, double *gram, hipStream_t stream);

/*
 * bkmoo_conflicts — per-bucket gradient-conflict diagnostics from Gram
 * matrices.  Two task gradients conflict when their inner product (their
 * cosine similarity) is negative (Section 2.1; the appendix definition of
 * conflicting gradients); Figure 1 follows the mean and standard deviation
 * of the pairwise cosines and counts a step as conflicting when some pair
 * is negative.  Reads only `gram` (B*K*K*8 bytes), one thread per bucket,
 * fp64, pairs i < j in lexicographic order.
 *
 *   gram     (in)  fp64 [B][K][K] (as written by bkmoo_gram / bkmoo_resolve)
 *   cosines  (out, may be NULL) fp64 [B][K][K], symmetric:
 *            G_ij / sqrt(G_ii G_jj) clipped to [-1, 1], 0 when either
 *            gradient is zero; diagonal 1 (0 for a zero gradient)
 *   summary  (out, may be NULL) fp64 [B][3]: mean, population standard
 *            deviation and minimum of the K(K-1)/2 pairwise cosines
 *   pairs    (out, may be NULL) int32 [B][3]: i, j (i < j) of the smallest
 *            cosine, the first pair on ties; the number of pairs with
 *            G_ij < 0 (> 0: the bucket has a conflict)
 *
 * A bucket whose Gram holds a NaN or infinity gets NaN cosines and summary
 * and pairs (-1, -1, -1).  All pointers are device pointers owned by the
 * caller; the call is asynchronous on `stream`.  BKMOO_EINVAL for K < 2,
 * B < 1, a null `gram` or all three outputs null; BKMOO_EUNSUPPORTED for
 * K > 16.
 */
bkmoo_status bkmoo_conflicts(int32_t K, int32_t B, const double *gram, double *cosines,
                             double *summary, int32_t *pairs, hipStream_t stream);

/*
 * bkmoo_resolve_traffic — the bytes a bkmoo_resolve call requests from
 * memory on `path` (*bytes, host) for these bucket offsets (host array,
 * int64 [B+1]): every gradient byte each pass reads plus the update written,
 * counted from the path's own data movement.  On the hybrid path part of the
 * second read of a streamed element may be served by the last-level cache,
 * so its HBM bytes can be lower:
 *   BKMOO_PATH_TWO_PASS  2*K*s*N + s_out*N
 *   BKMOO_PATH_HYBRID    K*s*N + s_out*N, plus K*s per element a data
 *                        workgroup did not keep on chip (read twice)
 * with s, s_out the input and output element sizes; BKMOO_PATH_REFILL as
 *                        BKMOO_PATH_HYBRID with its own (larger) kept share.  The small per-bucket
 * terms (offsets, Gram matrices, weights, partial sums) are left out.  The
 * hybrid path depends on the current device's CU count, and its segments
 * also on the method and iteration count (`method`,
 * `max_iter`, as given to bkmoo_resolve), which decide whether the first
 * workgroup of each CU takes a longer segment.  BKMOO_EINVAL
 * for bad sizes or pointers, invalid offsets, method or iteration count, or
 * an unknown path;
 * BKMOO_EUNSUPPORTED for the hybrid path with K > 8 or the refill path with
 * K > 10; BKMOO_EHIP when the
 * current device cannot be queried.
 */
bkmoo_status bkmoo_resolve_traffic(int32_t K, int64_t N, int32_t B, const int64_t *offsets_host,
                                   bkmoo_dtype dt, bkmoo_dtype out_dt, bkmoo_method method, int32_t max_iter,
                                   int32_t path, uint64_t *bytes);

/*
 * bkmoo_read_device_error — copy the workspace's device error word into
 * *err (host) after waiting for `stream`.  This call synchronises; it is a
 * diagnostic, not part of the hot path.  0 means the last call that used
 * this workspace found no error.
 */
bkmoo_status bkmoo_read_device_error(const void *workspace, uint32_t *err, hipStream_t stream);

/*
 * bkmoo_set_grid_override — number of workgroups the streaming kernels
 * launch (0 restores the automatic choice: enough to fill every CU).
 * Results do not depend on it; it exists for tuning and for tests of that
 * independence.  Process-wide setting.
 */
bkmoo_status bkmoo_set_grid_override(int32_t workgroups);

/*
 * bkmoo_resolve_path — the implementation bkmoo_resolve would use for these
 * arguments on the current device (*path, host): BKMOO_PATH_TWO_PASS,
 * BKMOO_PATH_HYBRID or BKMOO_PATH_REFILL.  `aligned` says whether every row and the output
 * start at the same 16-byte phase.
 */
bkmoo_status bkmoo_resolve_path(int32_t K, int64_t N, int32_t B, bkmoo_dtype dt, bkmoo_dtype out_dt,
                                int32_t aligned, bkmoo_method method, int32_t max_iter,
                                int32_t *path);

/*
 * bkmoo_set_resolve_path — force bkmoo_resolve's implementation
 * (0: automatic, BKMOO_PATH_TWO_PASS, or BKMOO_PATH_HYBRID or
 * BKMOO_PATH_REFILL when eligible: K <= 8 or K <= 10, aligned rows, not an
 * exact method; an ineligible call runs the two passes).  Process-wide; for
 * tests and tuning.  BKMOO_EINVAL for any other value.
 */
bkmoo_status bkmoo_set_resolve_path(int32_t path);

/*
 * bkmoo_set_wait_limit — polls of the cooperative paths' bounded waits (for
 * a bucket's arrivals or weights) before a workgroup gives up and sets
 * BKMOO_DEVERR_TIMEOUT
 * (default 4194304, about a second or more).  Process-wide; lets tests force
 * the timeout path from the host.  0 is rejected.
 */
bkmoo_status bkmoo_set_wait_limit(uint32_t polls);

/* Human-readable name of a status code (static string). */
const char *bkmoo_status_string(bkmoo_status st);

#ifdef __cplusplus
}
#endif

#endif /* BKMOO_H */
