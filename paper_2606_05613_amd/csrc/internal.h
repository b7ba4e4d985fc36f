// Internal declarations shared by the bkmoo translation units (not installed).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace bkmoo {

constexpr int kMinK = 2;
constexpr int kMaxK = 16;
constexpr int kExactMaxK = 10;  // exact solvers: 2^K - 1 supports per bucket
constexpr int kHybridMaxK = 8;  // the pipelined cooperative resolve (hybrid.hip)
constexpr int kThreads = 256;          // streaming kernels: 4 wavefronts of 64
constexpr int kWave = 64;

enum Dtype : int { F32 = 0, BF16 = 1 };

// Vectors of 16 bytes: 4 fp32 or 8 bf16 elements.
constexpr int vec_elems(int dt) { return dt == F32 ? 4 : 8; }
constexpr int elem_bytes(int dt) { return dt == F32 ? 4 : 2; }

// Streaming-pass shapes.  A chunk is U iterations of kThreads * R 16-byte
// vectors per task row; chunks never straddle buckets, so bucket b holds
// ceil(n_b / C) chunks.  K * R bounds the registers holding loaded data (4
// per vector) next to the pass's accumulators; occupancy supplies the rest
// of the memory-level parallelism.  The two passes are tuned separately
// (measured on MI355X): the Gram pass prefers long chunks (fewer fixed-order
// reductions), the combine pass shorter ones.  Above K = 4 one vector per
// row and iteration keeps the Gram kernel under 256 VGPRs (two wavefronts
// per SIMD instead of one at K = 8: 19.5 ms instead of 23.5 ms for 128 GB)
// and speeds the combine by 5%.  R * U is the same for every K <= 8, and a
// lane visits its vectors of a chunk in the same order for R = 1 and R = 2,
// so the Gram sums do not depend on the shape.  Each thread accumulates
// R * U * V elements of a chunk in fp32 in the Gram pass.
struct PassShape {
  int R, U;
};
constexpr PassShape gram_shape(int K) { return K <= 4 ? PassShape{2, 8} : PassShape{1, 16}; }
constexpr PassShape combine_shape(int K) { return K <= 4 ? PassShape{2, 4} : PassShape{1, 8}; }

constexpr int64_t shape_elems(PassShape p, int dt) {
  return (int64_t)kThreads * p.R * p.U * vec_elems(dt);
}
constexpr int64_t gram_chunk_elems(int K, int dt) { return shape_elems(gram_shape(K), dt); }
constexpr int64_t combine_chunk_elems(int K, int dt) { return shape_elems(combine_shape(K), dt); }

constexpr int pairs(int K) { return K * (K + 1) / 2; }

// The Gram finalize adds a bucket's chunk slots in groups of this many
// consecutive chunks (one workgroup per group), then the group sums in group
// order: the summation order depends only on the bucket's chunk count.
constexpr int kFinalizeGroup = 1024;

// Partial-Gram slots the workspace always has room for (the pipelined
// cooperative kernel uses two sets of one slot per workgroup that holds data).
constexpr int64_t kCoopSlots = 1024;

// The cooperative kernel's per-bucket arrival counters and flags sit 128
// bytes apart (one per cache line): with 4-byte neighbours, device-scope
// atomics on one bucket's counter and polls of the next buckets' counters
// contend for the same line (measured: 1.4 ms of a 23 ms step).
constexpr int64_t kSyncStride = 32;  // uint32 words
// Copies of each bucket's weights flag on the cooperative path: ~500 data
// workgroups poll it, and one copy (one line, one memory channel) per
// eighth of them keeps the polls from queueing on one channel.
constexpr int kFlagCopies = 8;

// Workspace layout (every region 256-byte aligned):
//   [0, 256)            header: uint32 error word at byte 0
//   chunk_start         int64 [B + 1]     (prefix sum of chunks per bucket)
//   gram                fp64  [B][K][K]   (used when the caller passes none)
//   weights             fp32  [B][K]      (used when the caller passes none)
//   partials            fp64  [cap][P]    cap = ceil(N / C) + B (at least kCoopSlots slots of P
//                                         rounded up to even)
//   group_start         int64 [B + 1]     (prefix sum of finalize groups per bucket)
//   groups              fp64  [gcap][P]   gcap = cap / kFinalizeGroup + B + 1
//   sync                uint32 [1 + kFlagCopies][B][kSyncStride]  cooperative path: arrival
//                       counters, then kFlagCopies copies of the flags
struct Layout {
  size_t err, chunk_start, gram, weights, partials, group_start, groups, sync, total;
  int64_t cap_chunks, cap_groups;
};

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

inline Layout layout(int K, int64_t N, int B, int dt) {
  Layout L;
  const int64_t C = gram_chunk_elems(K, dt);  // the smallest chunk with partial slots
  L.cap_chunks = (N + C - 1) / C + B;
  // at least two sets of slots for up to 512 workgroups of a cooperative kernel
  if (L.cap_chunks < kCoopSlots) L.cap_chunks = kCoopSlots;
  size_t o = 0;
  L.err = o;            o += 256;
  L.chunk_start = o;    o = align256(o + sizeof(int64_t) * (size_t)(B + 1));
  L.gram = o;           o = align256(o + sizeof(double) * (size_t)B * K * K);
  L.weights = o;        o = align256(o + sizeof(float) * (size_t)B * K);
  // (the single-buffer cooperative kernel pads each slot to an even count)
  const int64_t part = L.cap_chunks * pairs(K) > kCoopSlots * (pairs(K) + (pairs(K) & 1))
                           ? L.cap_chunks * pairs(K) : kCoopSlots * (pairs(K) + (pairs(K) & 1));
  L.partials = o;       o = align256(o + sizeof(double) * (size_t)part);
  L.cap_groups = L.cap_chunks / kFinalizeGroup + B + 1;
  L.group_start = o;    o = align256(o + sizeof(int64_t) * (size_t)(B + 1));
  L.groups = o;         o = align256(o + sizeof(double) * (size_t)L.cap_groups * pairs(K));
  L.sync = o;           o = align256(o + sizeof(uint32_t) * (1 + kFlagCopies) * (size_t)B * kSyncStride);
  L.total = o;
  return L;
}

constexpr uint32_t kErrOffsets = 0x1u;
constexpr uint32_t kErrTimeout = 0x2u;

// Pointers of the K task rows, passed by value as kernel arguments.
template <int K>
struct Rows {
  const void *p[K];
};

// ---- launchers (host) -------------------------------------------------------

struct StreamArgs {
  int K;
  int dt;                      // input dtype
  const void *const *rows;     // host array of K device pointers
  int64_t N;
  int B;
  const int64_t *offsets;      // device [B+1]
  const int64_t *chunk_start;  // device [B+1] (from the schedule kernel)
  const int64_t *group_start;  // device [B+1] finalize groups (Gram pass only)
  const uint32_t *err;         // device error word
  int shift;                   // rows are 16-byte aligned at element n = shift (mod V)
  bool vec;                    // 128-bit path allowed
  int grid;                    // workgroups (0: automatic)
};

// Validates offsets, writes chunk_start for chunks of C elements (and, if
// group_start is not null, the prefix of finalize groups), clears the error
// word and zeroes `nsync` words at `sync` (may be null).
hipError_t launch_schedule(const int64_t *offsets, int B, int64_t N, int64_t C, int64_t *chunk_start,
                           int64_t *group_start, uint32_t *err, uint32_t *sync, int64_t nsync,
                           hipStream_t s);
// Gram pass: per-chunk partials, group sums, then the per-bucket matrices.
// `cap_groups` bounds the number of finalize groups (sizes the group grid).
hipError_t launch_gram(const StreamArgs &a, double *partials, double *groups, int64_t cap_groups,
                       double *gram, hipStream_t s);
hipError_t launch_solve(int K, int B, const double *gram, int method, int max_iter, double c,
                        const int8_t *order, float *weights, double *aux, hipStream_t s);
hipError_t launch_combine(const StreamArgs &a, const float *weights, void *out, int out_dt,
                          hipStream_t s);
hipError_t launch_conflicts(int K, int B, const double *gram, double *cosines, double *summary,
                            int32_t *pairs, hipStream_t s);
// Bucket slices and the slice-order sum of partial Grams.
hipError_t launch_slice_offsets(const int64_t *offsets, int B, int T, int64_t *out, hipStream_t s);
hipError_t launch_gram_reduce(int K, int B, int T, const double *partial, int bucket_major, double *gram,
                              hipStream_t s);
// Exact MGDA / CAGrad solvers by support enumeration (K <= kExactMaxK).
hipError_t launch_exact_solve(int K, int B, const double *gram, int method, double c, float *weights,
                              double *aux, hipStream_t s);

// Pipelined, partly resident resolve (K <= kHybridMaxK): cooperative grid (0 if the
// combination cannot run this way), and how many of its workgroups hold data
// (the rest solve); partials must hold 2 * data workgroups slots.
int hybrid_grid(int K, int dt, int out_dt);
int hybrid_data_workgroups(int grid);
// Data workgroups dispatched first onto their CU (0 unless the grid is two
// workgroups per CU): the ones a segment skew gives more data.  The
// kHybridSolvers workgroups dispatched right after them are the second
// residents of the solvers' CUs.
int hybrid_older_workgroups(int grid);
constexpr int kHybridSolvers = 4;  // workgroups of the hybrid grid that reduce and solve

// Segment [lo, hi) (relative to the bucket start) of slot w in a bucket of n
// elements, over gd segment slots in whole units of `unit` elements, and
// the number nseg of non-empty segments, which are always slots 0 ..
// nseg-1.  skew_pm = 0: equal shares.  Otherwise the first `older` slots
// take (1 + skew_pm/1000) times an equal share (rounded up) and the others
// split the rest evenly.
__host__ __device__ inline void hybrid_segment(int64_t n, int w, int gd, int older, int skew_pm, int64_t unit,
                                               int64_t &lo, int64_t &hi, int64_t &nseg) {
  const int64_t nu = (n + unit - 1) / unit;
  int64_t s, e;
  if (skew_pm <= 0 || older <= 0 || older >= gd) {
    const int64_t c = (nu + gd - 1) / gd;
    s = (int64_t)w * c;
    e = s + c;
    nseg = c > 0 ? (nu + c - 1) / c : 0;
  } else {
    const int64_t co = (nu * (1000 + skew_pm) + (int64_t)gd * 1000 - 1) / ((int64_t)gd * 1000);
    const int64_t rest = nu - (int64_t)older * co;
    const int gy = gd - older;
    const int64_t cy = rest > 0 ? (rest + gy - 1) / gy : 0;
    s = w < older ? (int64_t)w * co : (int64_t)older * co + (int64_t)(w - older) * cy;
    e = w < older ? s + co : s + cy;
    nseg = co == 0 ? 0 : rest <= 0 ? (nu + co - 1) / co : older + (cy > 0 ? (rest + cy - 1) / cy : 0);
  }
  lo = s * unit < n ? s * unit : n;
  hi = e * unit < n ? e * unit : n;
}

// How one call spreads each bucket over the hybrid kernel's data
// workgroups.  Data workgroup w holds segment slot(w) of nslots (none when
// slot(w) < 0).  Without `light` the slots are the workgroups themselves;
// with it the solvers' CU mates (the kHybridSolvers workgroups after the
// `older` ones) hold none and leave their CU to the solve.  skew_pm as in
// hybrid_segment.  Shared by the kernel and the host's traffic count.
struct HybLayout {
  int nslots, older, skew_pm, light;
  __host__ __device__ int slot(int w) const {
    return !light || w < older ? w : w < older + kHybridSolvers ? -1 : w - kHybridSolvers;
  }
  // segment of slot s (s < 0: the empty one at the bucket's end)
  __host__ __device__ void segment(int64_t n, int s, int64_t unit, int64_t &lo, int64_t &hi,
                                   int64_t &nseg) const {
    hybrid_segment(n, s < 0 ? nslots : s, nslots, older, skew_pm, unit, lo, hi, nseg);
  }
};
// Elements of its segment a data workgroup keeps on chip per bucket, and the
// granule segment lengths are rounded up to.
int64_t hybrid_held_elems(int K, int dt, int out_dt);
int64_t hybrid_unit_elems(int dt);
hipError_t launch_hybrid(int K, int dt, int out_dt, const void *const *rows, const int64_t *offs, int B,
                         int shift, int method, int iters, double c, const int8_t *order, double *gram,
                         float *weights, double *aux, void *out, double *partials, uint32_t *arrive,
                         uint32_t *flags, uint32_t *err, uint32_t spin_limit, int grid,
                         const HybLayout &layout, hipStream_t s);

int device_cu_count();

// Resident workgroups of kThreads per CU for a kernel (at least 1).
template <typename Kern>
int occupancy(Kern kern) {
  int occ = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, kern, kThreads, 0) != hipSuccess || occ < 1)
    occ = 1;
  return occ;
}

}  // namespace bkmoo
